// backward.hip - C ABI of the compactor's backward pass (fp32): the gradient
// of <dC_k, C_k> + <dC_v, C_v> with respect to every compactor tensor of one
// layer (the training hot path without the base model and its loss; paper
// Section 2.4 and Appendix E).
//
// A forward pass that keeps its intermediates (the attention probabilities
// of every cross- and self-attention head included) is followed by the chain
// rule in reverse, step by step, each step one strided GEMM or one row-wise
// kernel of bwd.hpp, batched over the KV heads (the heads share every
// projection, so each weight gradient is one product over all rows).  The
// cross-attention logit path (q~, k~, their norms and rotations, S = q k^T)
// and its adjoint (dP, dS, dq, dk) run in fp64: the d_l logit scale
// multiplies their rounding into the attention weights.  Everything else is
// fp32 on MFMA.
#include "bwd.hpp"
#include "host.hpp"
#include "refine64.hpp"

namespace still {

namespace {

// Split-K partial buffer of the backward's long-contraction products: its
// capacity in elements (fp64: 64 MiB) and the current call's buffer (per
// host thread, set for the duration of run_backward).
constexpr long KSPLIT_CAP = 8l << 20;
static thread_local void* t_kpart = nullptr;

struct BPlan {
  size_t pq, invf_b, invf_c, X, Z;
  size_t Zc[8], Yc[8], rc[8], qt[8], qn[8], q[8], kt[8], kn[8], k[8], v[8], P[8], Hc[8];
  size_t Zs[8], Ys[8], rs[8], qst[8], qsn[8], qs[8], kst[8], ksn[8], ks[8], vs[8], Ps[8], Hs[8];
  size_t Zf[8], Yf[8], rf[8], g[8], u[8], a[8];
  size_t Zo, ro, dZ, dY, dH, dP, dq, dk, dv, dA, dU, dck;
  size_t csp;   // column-sum chunk partials (bias gradients)
  size_t kpart; // split-K partial sums of the long-contraction products
  size_t total;
};
constexpr int BWD_MAX_BLOCKS = 8;

BPlan make_bplan(const still_config* c, const Dims& m) {
  BPlan p;
  memset(&p, 0, sizeof p);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  const size_t Ht = (size_t)m.H * m.t, HN = (size_t)m.H * m.N;
  p.pq = take(8 * m.t);
  p.invf_b = take(8 * (m.d / 2));
  p.invf_c = take(8 * (m.dc / 2));
  p.X = take(4 * HN * m.d2);
  p.Z = take(4 * Ht * m.D);
  for (int b = 0; b < c->n_blocks; ++b) {
    if (c->cross_every_block || b == 0) {
      p.Zc[b] = take(4 * Ht * m.D);
      p.Yc[b] = take(4 * Ht * m.D);
      p.rc[b] = take(4 * Ht);
      p.qt[b] = take(8 * Ht * m.Ec);   // the logit path in fp64: q~, q, k~, k and their norms
      p.qn[b] = take(8 * Ht * m.nc);
      p.q[b] = take(8 * Ht * m.Ec);
      p.kt[b] = take(8 * HN * m.Ec);
      p.kn[b] = take(8 * HN * m.nc);
      p.k[b] = take(8 * HN * m.Ec);
      p.v[b] = take(4 * HN * m.Ec);
      p.P[b] = take(4 * (size_t)m.H * m.nc * m.t * m.N);
      p.Hc[b] = take(4 * Ht * m.Ec);
    }
    if (m.ns > 0) {
      p.Zs[b] = take(4 * Ht * m.D);
      p.Ys[b] = take(4 * Ht * m.D);
      p.rs[b] = take(4 * Ht);
      p.qst[b] = take(4 * Ht * m.Es);
      p.qsn[b] = take(4 * Ht * m.ns);
      p.qs[b] = take(4 * Ht * m.Es);
      p.kst[b] = take(4 * Ht * m.Es);
      p.ksn[b] = take(4 * Ht * m.ns);
      p.ks[b] = take(4 * Ht * m.Es);
      p.vs[b] = take(4 * Ht * m.Es);
      p.Ps[b] = take(4 * (size_t)m.H * m.ns * m.t * m.t);
      p.Hs[b] = take(4 * Ht * m.Es);
    }
    if (m.F > 0) {
      p.Zf[b] = take(4 * Ht * m.D);
      p.Yf[b] = take(4 * Ht * m.D);
      p.rf[b] = take(4 * Ht);
      p.g[b] = take(4 * Ht * m.F);
      p.u[b] = take(4 * Ht * m.F);
      p.a[b] = take(4 * Ht * m.F);
    }
  }
  p.Zo = take(4 * Ht * m.D);
  p.ro = take(4 * Ht);
  const size_t E = std::max<size_t>(m.Ec, m.Es);
  p.dZ = take(4 * Ht * m.D);
  p.dY = take(4 * Ht * m.D);
  p.dH = take(4 * Ht * E);
  // dP (also the forward's logits S) and dq, dk hold fp64 for cross-attention
  p.dP = take(8 * std::max<size_t>((size_t)m.H * m.nc * m.t * m.N, (size_t)m.H * std::max(m.ns, 1) * m.t * m.t));
  p.dq = take(8 * Ht * E);
  p.dk = take(8 * std::max<size_t>(HN * m.Ec, Ht * m.Es));
  p.dv = take(4 * std::max<size_t>(HN * m.Ec, Ht * m.Es));
  p.dA = take(4 * Ht * std::max(m.F, 1));
  p.dU = take(4 * Ht * std::max(m.F, 1));
  p.dck = take(4 * Ht * m.d);
  p.csp = take(8ul * COLSUM_CHUNKS * std::max(m.Ec, std::max(m.Es, 1)));
  p.kpart = take(8ul * KSPLIT_CAP);
  p.total = off + 256;
  return p;
}

// one operand of the strided GEMMs: element (row, k) at base + row * rs + k * ks
struct Op {
  const void* p;
  long rs, ks;
};
inline Op rowmaj(const void* p, long ld) { return {p, ld, 1}; }   // [rows][k], k contiguous
inline Op colmaj(const void* p, long ld) { return {p, 1, ld}; }   // element (r, k) at k * ld + r

// C (M x N, leading dimension ldc) (+)= A B^T, batched over nb1 x nb2 with
// element strides s?1 / s?2 per batch index.
struct Batch {
  int nb1 = 1, nb2 = 1;
  long sa1 = 0, sa2 = 0, sb1 = 0, sb2 = 0, sc1 = 0, sc2 = 0;
};

SgemmArgs gemm_args(int M, int N, int K, Op A, Op B, void* C, long ldc, bool acc, const float* bias, Batch bt,
                    float alpha) {
  SgemmArgs g;
  g.A = (const float*)A.p;
  g.B = (const float*)B.p;
  g.C = (float*)C;
  g.am = A.rs;
  g.ak = A.ks;
  g.sa1 = bt.sa1;
  g.sa2 = bt.sa2;
  g.bn = B.rs;
  g.bk = B.ks;
  g.sb1 = bt.sb1;
  g.sb2 = bt.sb2;
  g.ldc = ldc;
  g.sc1 = bt.sc1;
  g.sc2 = bt.sc2;
  g.M = M;
  g.N = N;
  g.K = K;
  g.nb2 = bt.nb2;
  g.alpha = alpha;
  g.accumulate = acc ? 1 : 0;
  g.ksplit = 0;
  g.part = nullptr;
  g.bias = bias;
  return g;
}

// Split-K for products with few output tiles and a long contraction (the
// weight gradients contract over all H N keys or H t latents): grid row z of
// a one-batch launch takes k in [z kc, (z + 1) kc) and stores raw partial
// sums in the call's split buffer (set by run_backward for its thread), which
// ksplit_reduce_kernel sums in order.  Returns the split count (1 = none).
inline int ksplit_count(int M, int N, int K, long batch) {
  if (!t_kpart || batch != 1 || K < 2048) return 1;
  const long tiles = (long)((M + 63) / 64) * ((N + 63) / 64);
  if (tiles >= 1024) return 1;
  long s = 2048 / tiles;
  s = std::min(s, (long)K / 1024);
  s = std::min(s, 16l);
  s = std::min(s, KSPLIT_CAP / ((long)M * N));
  return s >= 2 ? (int)s : 1;
}

// C = A B^T on the fp32 MFMA kernel (float operands and result)
hipError_t sgemm(hipStream_t st, int M, int N, int K, Op A, Op B, float* C, long ldc, bool acc,
                 const float* bias = nullptr, Batch bt = Batch(), float alpha = 1.f) {
  SgemmArgs g = gemm_args(M, N, K, A, B, C, ldc, acc, bias, bt, alpha);
  const int splits = ksplit_count(M, N, K, (long)bt.nb1 * bt.nb2);
  if (splits > 1) {
    g.ksplit = (int)((((long)K + splits - 1) / splits + 31) / 32 * 32);
    g.part = t_kpart;
  }
  const int nz = splits > 1 ? (int)(((long)K + g.ksplit - 1) / g.ksplit) : bt.nb1 * bt.nb2;
  const dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64), (unsigned)nz);
  const bool ak = A.ks == 1, bk = B.ks == 1;
  if (ak && bk) hipLaunchKernelGGL((sgemm_kernel<true, true>), grid, dim3(256), 0, st, g);
  else if (ak) hipLaunchKernelGGL((sgemm_kernel<true, false>), grid, dim3(256), 0, st, g);
  else if (bk) hipLaunchKernelGGL((sgemm_kernel<false, true>), grid, dim3(256), 0, st, g);
  else hipLaunchKernelGGL((sgemm_kernel<false, false>), grid, dim3(256), 0, st, g);
  if (splits > 1) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((ksplit_reduce_kernel<float, float>), dim3(grid1d((long)M * N)), dim3(256), 0, st,
                       (const float*)t_kpart, nz, M, N, (float*)C, ldc, (double)alpha, bias, acc ? 1 : 0);
  }
  return hipGetLastError();
}

// C = A B^T with fp64 accumulation; TA, TB, TC the operand and result types
template <class TA, class TB, class TC>
hipError_t dgemm(hipStream_t st, int M, int N, int K, Op A, Op B, TC* C, long ldc, bool acc,
                 const float* bias = nullptr, Batch bt = Batch()) {
  SgemmArgs g = gemm_args(M, N, K, A, B, C, ldc, acc, bias, bt, 1.f);
  const int splits = ksplit_count(M, N, K, (long)bt.nb1 * bt.nb2);
  if (splits > 1) {
    g.ksplit = (int)((((long)K + splits - 1) / splits + 31) / 32 * 32);
    g.part = t_kpart;
  }
  const int nz = splits > 1 ? (int)(((long)K + g.ksplit - 1) / g.ksplit) : bt.nb1 * bt.nb2;
  const dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64), (unsigned)nz);
  const TA* a = (const TA*)A.p;
  const TB* b = (const TB*)B.p;
  const bool ak = A.ks == 1, bk = B.ks == 1;
  if (ak && bk) hipLaunchKernelGGL((dgemm_kernel<true, true, TA, TB, TC>), grid, dim3(256), 0, st, g, a, b, C);
  else if (ak) hipLaunchKernelGGL((dgemm_kernel<true, false, TA, TB, TC>), grid, dim3(256), 0, st, g, a, b, C);
  else if (bk) hipLaunchKernelGGL((dgemm_kernel<false, true, TA, TB, TC>), grid, dim3(256), 0, st, g, a, b, C);
  else hipLaunchKernelGGL((dgemm_kernel<false, false, TA, TB, TC>), grid, dim3(256), 0, st, g, a, b, C);
  if (splits > 1) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((ksplit_reduce_kernel<double, TC>), dim3(grid1d((long)M * N)), dim3(256), 0, st,
                       (const double*)t_kpart, nz, M, N, C, ldc, 1.0, bias, acc ? 1 : 0);
  }
  return hipGetLastError();
}

inline dim3 rows4(long rows) { return dim3((unsigned)((rows + 3) / 4)); }

still_status run_backward(const still_config* cfg, const Dims& m, const BPlan& p, char* ws,
                          const still_layer_weights* w, const float* K, const float* V, const double* positions,
                          double theta, bool rerotate, const float* dCk, const float* dCv,
                          const still_layer_weights* gr, float* Ck, float* Cv, hipStream_t st) {
  const long Ht = (long)m.H * m.t, HN = (long)m.H * m.N;
  const int H = m.H, t = m.t, nc = m.nc, dc = m.dc, ns = m.ns, ds = m.ds, D = m.D, d = m.d, d2 = m.d2;
  const long Ec = m.Ec, Es = m.Es, F = m.F;
  const long N = m.N;
  struct KpartScope {   // the split buffer of this call, cleared on every return path
    explicit KpartScope(void* p) { t_kpart = p; }
    ~KpartScope() { t_kpart = nullptr; }
  } kpart_scope(ws + p.kpart);
  auto F32 = [&](size_t off) { return (float*)(ws + off); };
  auto F64 = [&](size_t off) { return (double*)(ws + off); };
  const double* pq = (const double*)(ws + p.pq);
  const double* invf_b = (const double*)(ws + p.invf_b);
  const double* invf_c = (const double*)(ws + p.invf_c);
  float* X = F32(p.X);
  float* Z = F32(p.Z);
  const float sc = cfg->logit_scale_cross != 0.f ? cfg->logit_scale_cross : (float)dc;
  const float ss = cfg->logit_scale_self != 0.f ? cfg->logit_scale_self : (float)ds;
  const float eps = cfg->rms_eps, l2e = cfg->l2_eps;
  auto copy = [&](const float* src, float* dst, long n) {
    hipLaunchKernelGGL(b_copy_kernel, dim3(grid1d(n)), dim3(256), 0, st, src, dst, n);
    return hipGetLastError();
  };
  auto colsum = [&](auto* dx, long rows, long ld, int wd, float* db) -> hipError_t {
    if (!db) return hipSuccess;
    typedef typename std::remove_const<typename std::remove_pointer<decltype(dx)>::type>::type T;
    double* part = (double*)(ws + p.csp);
    hipLaunchKernelGGL((b_colsum_part_kernel<T>), dim3((unsigned)((wd + 255) / 256), COLSUM_CHUNKS), dim3(256), 0, st,
                       (const T*)dx, rows, ld, wd, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(b_colsum_fin_kernel, dim3((unsigned)((wd + 255) / 256)), dim3(256), 0, st, (const double*)part,
                       COLSUM_CHUNKS, wd, db);
    return hipGetLastError();
  };
  auto W = [](const void* x) { return (const float*)x; };

  // ------------------------------------------------------------ forward
  hipLaunchKernelGGL(positions_kernel, dim3(1), dim3(256), 0, st, positions, N, t, (double*)pq, (double*)nullptr);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(inv_freq64_kernel, dim3((d / 2 + 255) / 256), dim3(256), 0, st, theta, d, (double*)invf_b);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(inv_freq64_kernel, dim3((dc / 2 + 255) / 256), dim3(256), 0, st, cfg->compactor_rope_base, dc,
                     (double*)invf_c);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(b_stage_x_kernel, dim3(grid1d(HN * (d / 2))), dim3(256), 0, st, K, V, positions, invf_b, HN, N,
                     d, X);
  HIP_TRY(hipGetLastError());
  HIP_TRY(copy(W(w->latents), Z, Ht * D));
  for (int b = 0; b < cfg->n_blocks; ++b) {
    const still_block_weights& bw = w->blocks[b];
    if (cfg->cross_every_block || b == 0) {
      float *Zc = F32(p.Zc[b]), *Yc = F32(p.Yc[b]), *rc = F32(p.rc[b]), *v = F32(p.v[b]);
      double *qt = F64(p.qt[b]), *qn = F64(p.qn[b]), *q = F64(p.q[b]), *kt = F64(p.kt[b]), *kn = F64(p.kn[b]);
      double* k = F64(p.k[b]);
      float *P = F32(p.P[b]), *Hc = F32(p.Hc[b]);
      double* S = F64(p.dP);
      HIP_TRY(copy(Z, Zc, Ht * D));
      hipLaunchKernelGGL(b_rms_fwd_kernel, rows4(Ht), dim3(256), 0, st, Z, Yc, rc, Ht, D, eps);
      HIP_TRY(hipGetLastError());
      HIP_TRY((dgemm<float, float, double>(st, (int)Ht, (int)Ec, D, rowmaj(Yc, D), rowmaj(bw.ca_wq, D), qt, Ec, false,
                                           W(bw.ca_bq))));
      hipLaunchKernelGGL((b_nrope_fwd_kernel<true, double>), rows4(Ht * nc), dim3(256), 0, st, qt, q, qn, Ht, nc, dc,
                         pq, (long)t, invf_c, l2e);
      HIP_TRY(hipGetLastError());
      HIP_TRY((dgemm<float, float, double>(st, (int)HN, (int)Ec, d2, rowmaj(X, d2), rowmaj(bw.ca_wk, d2), kt, Ec,
                                           false, W(bw.ca_bk))));
      hipLaunchKernelGGL((b_nrope_fwd_kernel<true, double>), rows4(HN * nc), dim3(256), 0, st, kt, k, kn, HN, nc, dc,
                         positions, N, invf_c, l2e);
      HIP_TRY(hipGetLastError());
      HIP_TRY(sgemm(st, (int)HN, (int)Ec, d2, rowmaj(X, d2), rowmaj(bw.ca_wv, d2), v, Ec, false));
      Batch hc;   // per (KV head h, cross head c)
      hc.nb1 = H;
      hc.nb2 = nc;
      // S = q k^T  [t][N]
      Batch s1 = hc;
      s1.sa1 = t * Ec, s1.sa2 = dc, s1.sb1 = N * Ec, s1.sb2 = dc, s1.sc1 = nc * t * N, s1.sc2 = t * N;
      HIP_TRY((dgemm<double, double, double>(st, t, (int)N, dc, rowmaj(q, Ec), rowmaj(k, Ec), S, N, false, nullptr,
                                             s1)));
      hipLaunchKernelGGL((b_softmax_fwd_kernel<double>), rows4((long)H * nc * t), dim3(256), 0, st, S, P,
                         (long)H * nc * t, (int)N, sc);
      HIP_TRY(hipGetLastError());
      // head = P v  [t][dc]
      Batch s2 = hc;
      s2.sa1 = nc * t * N, s2.sa2 = t * N, s2.sb1 = N * Ec, s2.sb2 = dc, s2.sc1 = t * Ec, s2.sc2 = dc;
      HIP_TRY(sgemm(st, t, dc, (int)N, rowmaj(P, N), colmaj(v, Ec), Hc, Ec, false, nullptr, s2));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)Ec, rowmaj(Hc, Ec), rowmaj(bw.ca_wo, Ec), Z, D, true));
    }
    if (ns > 0) {
      float *Zs = F32(p.Zs[b]), *Ys = F32(p.Ys[b]), *rs = F32(p.rs[b]), *qst = F32(p.qst[b]), *qsn = F32(p.qsn[b]);
      float *qs = F32(p.qs[b]), *kst = F32(p.kst[b]), *ksn = F32(p.ksn[b]), *ks = F32(p.ks[b]), *vs = F32(p.vs[b]);
      float *Ps = F32(p.Ps[b]), *Hs = F32(p.Hs[b]);
      HIP_TRY(copy(Z, Zs, Ht * D));
      hipLaunchKernelGGL(b_rms_fwd_kernel, rows4(Ht), dim3(256), 0, st, Z, Ys, rs, Ht, D, eps);
      HIP_TRY(hipGetLastError());
      HIP_TRY(sgemm(st, (int)Ht, (int)Es, D, rowmaj(Ys, D), rowmaj(bw.sa_wq, D), qst, Es, false, W(bw.sa_bq)));
      HIP_TRY(sgemm(st, (int)Ht, (int)Es, D, rowmaj(Ys, D), rowmaj(bw.sa_wk, D), kst, Es, false, W(bw.sa_bk)));
      HIP_TRY(sgemm(st, (int)Ht, (int)Es, D, rowmaj(Ys, D), rowmaj(bw.sa_wv, D), vs, Es, false));
      hipLaunchKernelGGL((b_nrope_fwd_kernel<true>), rows4(Ht * ns), dim3(256), 0, st, qst, qs, qsn, Ht, ns, ds,
                         (const double*)nullptr, 1L, (const double*)nullptr, l2e);
      HIP_TRY(hipGetLastError());
      hipLaunchKernelGGL((b_nrope_fwd_kernel<true>), rows4(Ht * ns), dim3(256), 0, st, kst, ks, ksn, Ht, ns, ds,
                         (const double*)nullptr, 1L, (const double*)nullptr, l2e);
      HIP_TRY(hipGetLastError());
      Batch s1;
      s1.nb1 = H, s1.nb2 = ns;
      s1.sa1 = t * Es, s1.sa2 = ds, s1.sb1 = t * Es, s1.sb2 = ds, s1.sc1 = (long)ns * t * t, s1.sc2 = (long)t * t;
      HIP_TRY(sgemm(st, t, t, ds, rowmaj(qs, Es), rowmaj(ks, Es), Ps, t, false, nullptr, s1));
      hipLaunchKernelGGL((b_softmax_fwd_kernel<float>), rows4((long)H * ns * t), dim3(256), 0, st, Ps, Ps,
                         (long)H * ns * t, t, ss);
      HIP_TRY(hipGetLastError());
      Batch s2;
      s2.nb1 = H, s2.nb2 = ns;
      s2.sa1 = (long)ns * t * t, s2.sa2 = (long)t * t, s2.sb1 = t * Es, s2.sb2 = ds, s2.sc1 = t * Es, s2.sc2 = ds;
      HIP_TRY(sgemm(st, t, ds, t, rowmaj(Ps, t), colmaj(vs, Es), Hs, Es, false, nullptr, s2));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)Es, rowmaj(Hs, Es), rowmaj(bw.sa_wo, Es), Z, D, true));
    }
    if (F > 0) {
      float *Zf = F32(p.Zf[b]), *Yf = F32(p.Yf[b]), *rf = F32(p.rf[b]), *g = F32(p.g[b]), *u = F32(p.u[b]);
      float* a = F32(p.a[b]);
      const bool glu = cfg->ffn_kind == STILL_FFN_SWIGLU;
      HIP_TRY(copy(Z, Zf, Ht * D));
      hipLaunchKernelGGL(b_rms_fwd_kernel, rows4(Ht), dim3(256), 0, st, Z, Yf, rf, Ht, D, eps);
      HIP_TRY(hipGetLastError());
      if (glu) HIP_TRY(sgemm(st, (int)Ht, (int)F, D, rowmaj(Yf, D), rowmaj(bw.ffn_wg, D), g, F, false));
      HIP_TRY(sgemm(st, (int)Ht, (int)F, D, rowmaj(Yf, D), rowmaj(bw.ffn_wu, D), u, F, false));
      hipLaunchKernelGGL(b_act_fwd_kernel, dim3(grid1d(Ht * F)), dim3(256), 0, st, g, u, a, Ht * F, glu ? 1 : 0);
      HIP_TRY(hipGetLastError());
      HIP_TRY(sgemm(st, (int)Ht, D, (int)F, rowmaj(a, F), rowmaj(bw.ffn_wd, F), Z, D, true));
    }
  }
  float* Zo = Z;
  if (cfg->final_norm) {
    Zo = F32(p.Zo);
    hipLaunchKernelGGL(b_rms_fwd_kernel, rows4(Ht), dim3(256), 0, st, Z, Zo, F32(p.ro), Ht, D, eps);
    HIP_TRY(hipGetLastError());
  }
  if (Ck) {   // forward outputs, on request
    HIP_TRY(sgemm(st, (int)Ht, d, D, rowmaj(Zo, D), rowmaj(w->w_key, D), Ck, d, false));
    if (rerotate) {
      hipLaunchKernelGGL((b_nrope_fwd_kernel<false>), rows4(Ht), dim3(256), 0, st, Ck, Ck, (float*)nullptr, Ht, 1, d,
                         pq, (long)t, invf_b, l2e);
      HIP_TRY(hipGetLastError());
    }
  }
  if (Cv) HIP_TRY(sgemm(st, (int)Ht, d, D, rowmaj(Zo, D), rowmaj(w->w_val, D), Cv, d, false));

  // ------------------------------------------------------------ backward
  float *dZ = F32(p.dZ), *dY = F32(p.dY), *dH = F32(p.dH), *dP = F32(p.dP), *dq = F32(p.dq), *dk = F32(p.dk);
  float *dv = F32(p.dv), *dA = F32(p.dA), *dU = F32(p.dU), *dck = F32(p.dck);
  auto G = [](const void* x) { return (float*)x; };
  // output heads: C_k = R(p_q) (Zo W_key^T), C_v = Zo W_val^T
  if (rerotate) {
    hipLaunchKernelGGL((b_nrope_bwd_kernel<false>), rows4(Ht), dim3(256), 0, st, (const float*)nullptr,
                       (const float*)nullptr, dCk, dck, Ht, 1, d, pq, (long)t, invf_b, l2e);
    HIP_TRY(hipGetLastError());
  } else {
    HIP_TRY(copy(dCk, dck, Ht * d));
  }
  if (gr->w_key) HIP_TRY(sgemm(st, d, D, (int)Ht, colmaj(dck, d), colmaj(Zo, D), G(gr->w_key), D, false));
  if (gr->w_val) HIP_TRY(sgemm(st, d, D, (int)Ht, colmaj(dCv, d), colmaj(Zo, D), G(gr->w_val), D, false));
  float* dZo = cfg->final_norm ? dY : dZ;
  HIP_TRY(sgemm(st, (int)Ht, D, d, rowmaj(dck, d), colmaj(w->w_key, D), dZo, D, false));
  HIP_TRY(sgemm(st, (int)Ht, D, d, rowmaj(dCv, d), colmaj(w->w_val, D), dZo, D, true));
  if (cfg->final_norm) {
    hipLaunchKernelGGL(b_fill_kernel, dim3(grid1d(Ht * D)), dim3(256), 0, st, dZ, Ht * D, 0.f);
    HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(b_rms_bwd_kernel, rows4(Ht), dim3(256), 0, st, Z, dY, F32(p.ro), dZ, Ht, D);
    HIP_TRY(hipGetLastError());
  }
  for (int b = cfg->n_blocks - 1; b >= 0; --b) {
    const still_block_weights& bw = w->blocks[b];
    const still_block_weights& gb = gr->blocks[b];
    if (F > 0) {
      float *Zf = F32(p.Zf[b]), *Yf = F32(p.Yf[b]), *rf = F32(p.rf[b]), *g = F32(p.g[b]), *u = F32(p.u[b]);
      float* a = F32(p.a[b]);
      const bool glu = cfg->ffn_kind == STILL_FFN_SWIGLU;
      if (gb.ffn_wd) HIP_TRY(sgemm(st, D, (int)F, (int)Ht, colmaj(dZ, D), colmaj(a, F), G(gb.ffn_wd), F, false));
      HIP_TRY(sgemm(st, (int)Ht, (int)F, D, rowmaj(dZ, D), colmaj(bw.ffn_wd, F), dA, F, false));
      // dg over da (same index, same thread), du separately
      hipLaunchKernelGGL(b_act_bwd_kernel, dim3(grid1d(Ht * F)), dim3(256), 0, st, g, u, dA, dA, dU, Ht * F,
                         glu ? 1 : 0);
      HIP_TRY(hipGetLastError());
      if (glu && gb.ffn_wg) HIP_TRY(sgemm(st, (int)F, D, (int)Ht, colmaj(dA, F), colmaj(Yf, D), G(gb.ffn_wg), D, false));
      if (gb.ffn_wu) HIP_TRY(sgemm(st, (int)F, D, (int)Ht, colmaj(dU, F), colmaj(Yf, D), G(gb.ffn_wu), D, false));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)F, rowmaj(dU, F), colmaj(bw.ffn_wu, D), dY, D, false));
      if (glu) HIP_TRY(sgemm(st, (int)Ht, D, (int)F, rowmaj(dA, F), colmaj(bw.ffn_wg, D), dY, D, true));
      hipLaunchKernelGGL(b_rms_bwd_kernel, rows4(Ht), dim3(256), 0, st, Zf, dY, rf, dZ, Ht, D);
      HIP_TRY(hipGetLastError());
    }
    if (ns > 0) {
      float *Zs = F32(p.Zs[b]), *Ys = F32(p.Ys[b]), *rs = F32(p.rs[b]), *qst = F32(p.qst[b]), *qsn = F32(p.qsn[b]);
      float *qs = F32(p.qs[b]), *kst = F32(p.kst[b]), *ksn = F32(p.ksn[b]), *ks = F32(p.ks[b]), *vs = F32(p.vs[b]);
      float *Ps = F32(p.Ps[b]), *Hs = F32(p.Hs[b]);
      if (gb.sa_wo) HIP_TRY(sgemm(st, D, (int)Es, (int)Ht, colmaj(dZ, D), colmaj(Hs, Es), G(gb.sa_wo), Es, false));
      HIP_TRY(sgemm(st, (int)Ht, (int)Es, D, rowmaj(dZ, D), colmaj(bw.sa_wo, Es), dH, Es, false));
      Batch hb;
      hb.nb1 = H, hb.nb2 = ns;
      // dv = P^T dH   [t][ds]
      Batch b1 = hb;
      b1.sa1 = (long)ns * t * t, b1.sa2 = (long)t * t, b1.sb1 = t * Es, b1.sb2 = ds, b1.sc1 = t * Es, b1.sc2 = ds;
      HIP_TRY(sgemm(st, t, ds, t, colmaj(Ps, t), colmaj(dH, Es), dv, Es, false, nullptr, b1));
      // dP = dH v^T   [t][t]
      Batch b2 = hb;
      b2.sa1 = t * Es, b2.sa2 = ds, b2.sb1 = t * Es, b2.sb2 = ds, b2.sc1 = (long)ns * t * t, b2.sc2 = (long)t * t;
      HIP_TRY(sgemm(st, t, t, ds, rowmaj(dH, Es), rowmaj(vs, Es), dP, t, false, nullptr, b2));
      hipLaunchKernelGGL((b_softmax_bwd_kernel<float>), rows4((long)H * ns * t), dim3(256), 0, st, Ps, dP,
                         (long)H * ns * t, t, ss);
      HIP_TRY(hipGetLastError());
      // dq = dS k, dk = dS^T q   [t][ds]
      Batch b3 = hb;
      b3.sa1 = (long)ns * t * t, b3.sa2 = (long)t * t, b3.sb1 = t * Es, b3.sb2 = ds, b3.sc1 = t * Es, b3.sc2 = ds;
      HIP_TRY(sgemm(st, t, ds, t, rowmaj(dP, t), colmaj(ks, Es), dq, Es, false, nullptr, b3));
      HIP_TRY(sgemm(st, t, ds, t, colmaj(dP, t), colmaj(qs, Es), dk, Es, false, nullptr, b3));
      hipLaunchKernelGGL((b_nrope_bwd_kernel<true>), rows4(Ht * ns), dim3(256), 0, st, qst, qsn, dq, dq, Ht, ns, ds,
                         (const double*)nullptr, 1L, (const double*)nullptr, l2e);
      HIP_TRY(hipGetLastError());
      hipLaunchKernelGGL((b_nrope_bwd_kernel<true>), rows4(Ht * ns), dim3(256), 0, st, kst, ksn, dk, dk, Ht, ns, ds,
                         (const double*)nullptr, 1L, (const double*)nullptr, l2e);
      HIP_TRY(hipGetLastError());
      if (gb.sa_wq) HIP_TRY(sgemm(st, (int)Es, D, (int)Ht, colmaj(dq, Es), colmaj(Ys, D), G(gb.sa_wq), D, false));
      if (gb.sa_wk) HIP_TRY(sgemm(st, (int)Es, D, (int)Ht, colmaj(dk, Es), colmaj(Ys, D), G(gb.sa_wk), D, false));
      if (gb.sa_wv) HIP_TRY(sgemm(st, (int)Es, D, (int)Ht, colmaj(dv, Es), colmaj(Ys, D), G(gb.sa_wv), D, false));
      HIP_TRY(colsum((const float*)dq, Ht, Es, (int)Es, G(gb.sa_bq)));
      HIP_TRY(colsum((const float*)dk, Ht, Es, (int)Es, G(gb.sa_bk)));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)Es, rowmaj(dq, Es), colmaj(bw.sa_wq, D), dY, D, false));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)Es, rowmaj(dk, Es), colmaj(bw.sa_wk, D), dY, D, true));
      HIP_TRY(sgemm(st, (int)Ht, D, (int)Es, rowmaj(dv, Es), colmaj(bw.sa_wv, D), dY, D, true));
      hipLaunchKernelGGL(b_rms_bwd_kernel, rows4(Ht), dim3(256), 0, st, Zs, dY, rs, dZ, Ht, D);
      HIP_TRY(hipGetLastError());
    }
    if (cfg->cross_every_block || b == 0) {
      float *Zc = F32(p.Zc[b]), *Yc = F32(p.Yc[b]), *rc = F32(p.rc[b]), *v = F32(p.v[b]);
      double *qt = F64(p.qt[b]), *qn = F64(p.qn[b]), *q = F64(p.q[b]), *kt = F64(p.kt[b]), *kn = F64(p.kn[b]);
      double* k = F64(p.k[b]);
      float *P = F32(p.P[b]), *Hc = F32(p.Hc[b]);
      double *dP64 = F64(p.dP), *dq64 = F64(p.dq), *dk64 = F64(p.dk);
      if (gb.ca_wo) HIP_TRY(sgemm(st, D, (int)Ec, (int)Ht, colmaj(dZ, D), colmaj(Hc, Ec), G(gb.ca_wo), Ec, false));
      HIP_TRY(sgemm(st, (int)Ht, (int)Ec, D, rowmaj(dZ, D), colmaj(bw.ca_wo, Ec), dH, Ec, false));
      Batch hc;
      hc.nb1 = H, hc.nb2 = nc;
      // dv = P^T dH   [N][dc]
      Batch b1 = hc;
      b1.sa1 = nc * t * N, b1.sa2 = t * N, b1.sb1 = t * Ec, b1.sb2 = dc, b1.sc1 = N * Ec, b1.sc2 = dc;
      HIP_TRY(sgemm(st, (int)N, dc, t, colmaj(P, N), colmaj(dH, Ec), dv, Ec, false, nullptr, b1));
      // dP = dH v^T   [t][N]
      Batch b2 = hc;
      b2.sa1 = t * Ec, b2.sa2 = dc, b2.sb1 = N * Ec, b2.sb2 = dc, b2.sc1 = nc * t * N, b2.sc2 = t * N;
      HIP_TRY((dgemm<float, float, double>(st, t, (int)N, dc, rowmaj(dH, Ec), rowmaj(v, Ec), dP64, N, false, nullptr,
                                           b2)));
      hipLaunchKernelGGL((b_softmax_bwd_kernel<double>), rows4((long)H * nc * t), dim3(256), 0, st, P, dP64,
                         (long)H * nc * t, (int)N, sc);
      HIP_TRY(hipGetLastError());
      // dq = dS k   [t][dc]
      Batch b3 = hc;
      b3.sa1 = nc * t * N, b3.sa2 = t * N, b3.sb1 = N * Ec, b3.sb2 = dc, b3.sc1 = t * Ec, b3.sc2 = dc;
      HIP_TRY((dgemm<double, double, double>(st, t, dc, (int)N, rowmaj(dP64, N), colmaj(k, Ec), dq64, Ec, false,
                                             nullptr, b3)));
      // dk = dS^T q   [N][dc]
      Batch b4 = hc;
      b4.sa1 = nc * t * N, b4.sa2 = t * N, b4.sb1 = t * Ec, b4.sb2 = dc, b4.sc1 = N * Ec, b4.sc2 = dc;
      HIP_TRY((dgemm<double, double, double>(st, (int)N, dc, t, colmaj(dP64, N), colmaj(q, Ec), dk64, Ec, false,
                                             nullptr, b4)));
      hipLaunchKernelGGL((b_nrope_bwd_kernel<true, double>), rows4(Ht * nc), dim3(256), 0, st, qt, qn, dq64, dq64, Ht,
                         nc, dc, pq, (long)t, invf_c, l2e);
      HIP_TRY(hipGetLastError());
      hipLaunchKernelGGL((b_nrope_bwd_kernel<true, double>), rows4(HN * nc), dim3(256), 0, st, kt, kn, dk64, dk64, HN,
                         nc, dc, positions, N, invf_c, l2e);
      HIP_TRY(hipGetLastError());
      if (gb.ca_wq)
        HIP_TRY((dgemm<double, float, float>(st, (int)Ec, D, (int)Ht, colmaj(dq64, Ec), colmaj(Yc, D), G(gb.ca_wq), D,
                                             false)));
      if (gb.ca_wk)
        HIP_TRY((dgemm<double, float, float>(st, (int)Ec, d2, (int)HN, colmaj(dk64, Ec), colmaj(X, d2), G(gb.ca_wk),
                                             d2, false)));
      if (gb.ca_wv) HIP_TRY(sgemm(st, (int)Ec, d2, (int)HN, colmaj(dv, Ec), colmaj(X, d2), G(gb.ca_wv), d2, false));
      HIP_TRY(colsum((const double*)dq64, Ht, Ec, (int)Ec, G(gb.ca_bq)));
      HIP_TRY(colsum((const double*)dk64, HN, Ec, (int)Ec, G(gb.ca_bk)));
      HIP_TRY((dgemm<double, float, float>(st, (int)Ht, D, (int)Ec, rowmaj(dq64, Ec), colmaj(bw.ca_wq, D), dY, D,
                                           false)));
      hipLaunchKernelGGL(b_rms_bwd_kernel, rows4(Ht), dim3(256), 0, st, Zc, dY, rc, dZ, Ht, D);
      HIP_TRY(hipGetLastError());
    }
  }
  if (gr->latents) HIP_TRY(copy(dZ, G(gr->latents), Ht * D));
  return STILL_OK;
}

}  // namespace

}  // namespace still

using namespace still;

extern "C" {

size_t still_backward_workspace_size(const still_config* cfg, int64_t N, int32_t t) {
  Dims m;
  const std::string keep = g_last_error;
  if (make_dims(cfg, N, t, &m) != STILL_OK || !m.fp32 || cfg->n_blocks > BWD_MAX_BLOCKS) {
    g_last_error = keep;
    return 0;
  }
  return make_bplan(cfg, m).total;
}

still_status still_compact_layer_backward(const still_config* cfg, const still_layer_weights* w, const void* K,
                                          const void* V, const double* positions, int64_t N, double rope_theta,
                                          int32_t t, uint32_t flags, const void* dC_k, const void* dC_v,
                                          const still_layer_weights* grad, void* C_k, void* C_v, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  Dims m;
  still_status s = make_dims(cfg, N, t, &m);
  if (s != STILL_OK) return s;
  if (!m.fp32) return fail(STILL_E_UNSUPPORTED, "the backward pass runs in STILL_MODE_FP32 only");
  if (cfg->n_blocks > BWD_MAX_BLOCKS) return fail(STILL_E_UNSUPPORTED, "backward supports up to %d blocks", BWD_MAX_BLOCKS);
  if (flags & ~(uint32_t)STILL_F_REROTATE) return fail(STILL_E_INVAL, "unknown flags 0x%x", flags);
  if (!(rope_theta > 0.0)) return fail(STILL_E_INVAL, "rope_theta must be > 0");
  if (!positions || ((uintptr_t)positions & 7u)) return fail(STILL_E_INVAL, "positions NULL or misaligned");
  if ((s = check_layer(cfg, m, w, 0)) != STILL_OK) return s;
  if (!grad || !grad->blocks) return fail(STILL_E_INVAL, "gradient struct or its blocks array is NULL");
  if (grad->t_bank != t) return fail(STILL_E_SHAPE, "gradient latent bank %d != t %d", grad->t_bank, t);
  for (const void* q : {K, V, dC_k, dC_v})
    if (!q || ((uintptr_t)q & 15u)) return fail(STILL_E_INVAL, "K, V, dC_k, dC_v must be non-NULL, 16-byte aligned");
  for (const void* q : {(const void*)C_k, (const void*)C_v})
    if (q && ((uintptr_t)q & 15u)) return fail(STILL_E_INVAL, "C_k / C_v must be 16-byte aligned");
  const BPlan p = make_bplan(cfg, m);
  if (!workspace) return fail(STILL_E_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < p.total)
    return fail(STILL_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, p.total);
  char* ws = (char*)(((uintptr_t)workspace + 255) & ~(uintptr_t)255);
  hipStream_t st = (hipStream_t)stream;
  (void)hipGetLastError();
  return run_backward(cfg, m, p, ws, w, (const float*)K, (const float*)V, positions, rope_theta,
                      (flags & STILL_F_REROTATE) != 0, (const float*)dC_k, (const float*)dC_v, grad, (float*)C_k,
                      (float*)C_v, st);
}

}  // extern "C"
