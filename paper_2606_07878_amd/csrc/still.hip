// still.hip - C ABI (include/still.h) of the Still compactor forward pass on
// MI355X: argument validation, workspace planning and the per-layer launch
// sequence of the HIP kernels in gemm.hpp, attn.hpp and misc.hpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/still.h"
#include "attn.hpp"
#include "common.hpp"
#include "consumer.hpp"
#include "gemm.hpp"
#include "kproj.hpp"
#include "misc.hpp"
#include "refine.hpp"

namespace still {

static thread_local std::string g_last_error;

static still_status fail(still_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

#define HIP_TRY(expr)                                                                         \
  do {                                                                                        \
    hipError_t _e = (expr);                                                                   \
    if (_e != hipSuccess) return fail(STILL_E_HIP, "%s: %s", #expr, hipGetErrorString(_e));   \
  } while (0)

static inline long rup(long x, long m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------------------
// Optional per-class kernel timing with hipEvent pairs on the launch stream.
// ---------------------------------------------------------------------------
namespace timing {
struct Rec {
  int cls;
  hipEvent_t a, b;
};
static unsigned mask = 0;   // bit c: record launches of class c
static std::vector<Rec> pending;
static std::vector<hipEvent_t> spare;
static double ms[STILL_K_COUNT];
static long long count[STILL_K_COUNT];

static hipEvent_t get_event() {
  if (!spare.empty()) {
    hipEvent_t e = spare.back();
    spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Fold the oldest `n` pending records into the totals (waits for them).
static hipError_t harvest(size_t n) {
  if (n > pending.size()) n = pending.size();
  for (size_t i = 0; i < n; ++i) {
    Rec& r = pending[i];
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return e;
    float t = 0.f;
    e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess) return e;
    ms[r.cls] += t;
    count[r.cls] += 1;
    spare.push_back(r.a);
    spare.push_back(r.b);
  }
  pending.erase(pending.begin(), pending.begin() + n);
  return hipSuccess;
}

struct Scope {
  int cls;
  hipStream_t st;
  hipEvent_t a = nullptr;
  Scope(int c, hipStream_t s) : cls(c), st(s) {
    if (!(mask & (1u << c))) return;
    if (pending.size() >= 8192) harvest(4096);
    a = get_event();
    if (a) hipEventRecord(a, st);
  }
  ~Scope() {
    if (!a) return;
    hipEvent_t b = get_event();
    if (!b) return;
    hipEventRecord(b, st);
    pending.push_back({cls, a, b});
  }
};
}  // namespace timing

#define TIMED(cls) timing::Scope _timed_scope_##__LINE__((cls), st)

constexpr int GEMM_BN = 128;   // column tile of every GEMM (two halves of 64 pairs)
constexpr int ATT_TT = 128;    // latents per attention workgroup
constexpr int ATT_NB = 64;     // keys per attention block
constexpr int ATT_TOPK = 4;    // keys tracked per latent half-lane for logit refinement (fp32 kernel)
constexpr int XATT_KB = 256;   // keys per block of the fp16 cross-attention kernel
constexpr int XATT_TOPK = 4;   // keys tracked per (latent, wave, lane half) by the fp16 kernel
constexpr int REFINE_R = 4;    // keys per latent whose logits are recomputed accurately
static_assert(REFINE_R <= 8, "merge_kernel handles up to 8 refined keys per latent");
// waves of the fp16 cross-attention workgroup for a value width d2 = 2d
constexpr int xatt_waves(int) { return 4; }

// ---------------------------------------------------------------------------
// Derived dimensions and workspace layout
// ---------------------------------------------------------------------------
struct Dims {
  int H, d, D, d2, nc, dc, ns, ds, F, Ec, Es, t, tpad;
  long N, Npad;
  int np_c, np_s;       // sum-of-squares partials per (row, head)
  int topk, R;          // logit refinement
  int ncand;            // candidate keys per (split, latent row) written by the attention kernel
  int att_tt;           // latents per attention workgroup
  int splits;           // split-N factor of the cross-attention
  long keys_per_split;
  size_t cs;            // bytes of the compute/storage type
  bool fp32;
};

struct Plan {
  size_t pq, tab_ck, tab_cq, tab_bk, tab_bq;
  size_t wconv;          // bf16 mode: the layer's weight matrices converted to fp16
  size_t wkt;            // bf16 mode: fragment-tiled fp16 copy of the cross-attention W_K
  size_t X, XT, Z, Y, q, partq, rq, O;
  size_t Ylo, qex, cval, cidx, ridx, rval, Xc, rpart, crow, ccount;   // logit refinement
  // union region: cross-attention key side ...
  size_t k, partk, rk, opart, mpart, lpart;
  // ... or self-attention / FFN buffers
  size_t qs, ks, vT, partqs, partks, rqs, rks, Ssa, Psa, Osa, hid;
  size_t total;
};

static int key_block(const Dims& m) { return m.fp32 ? ATT_NB : XATT_KB; }

static int choose_splits(const Dims& m) {
  const long wgs = (long)((m.t + m.att_tt - 1) / m.att_tt) * m.H * m.nc;
  const long nblocks = (m.N + key_block(m) - 1) / key_block(m);
  // fp16 kernel: one workgroup per CU, aim for >= 2 per CU; fp32: >= 4
  long s = ((m.fp32 ? 1024 : 512) + wgs - 1) / wgs;
  if (s > nblocks) s = nblocks;
  if (s < 1) s = 1;
  return (int)s;
}

static still_status make_dims(const still_config* c, int64_t N, int32_t t, Dims* m) {
  if (!c) return fail(STILL_E_INVAL, "config is NULL");
  if (c->mode != STILL_MODE_BF16 && c->mode != STILL_MODE_FP32) return fail(STILL_E_DTYPE, "unknown mode %d", c->mode);
  if (c->n_kv_heads < 1 || c->head_dim < 2 || c->latent_dim < 1 || c->n_blocks < 1)
    return fail(STILL_E_INVAL, "non-positive dimension in config");
  if (N < 1 || t < 1) return fail(STILL_E_INVAL, "N and t must be >= 1 (N=%lld t=%d)", (long long)N, t);
  if (c->head_dim % 2) return fail(STILL_E_SHAPE, "head_dim must be even (got %d)", c->head_dim);
  if (c->n_cross_heads < 1) return fail(STILL_E_INVAL, "n_cross_heads must be >= 1");
  if (c->n_self_heads < 0) return fail(STILL_E_INVAL, "n_self_heads must be >= 0");
  if (c->ffn_kind < 0 || c->ffn_kind > 2) return fail(STILL_E_INVAL, "unknown ffn_kind %d", c->ffn_kind);
  if (c->ffn_kind != STILL_FFN_NONE && c->ffn_hidden < 1) return fail(STILL_E_INVAL, "ffn_hidden must be >= 1");
  if (!(c->compactor_rope_base > 0.0)) return fail(STILL_E_INVAL, "compactor_rope_base must be > 0");
  if (!(c->l2_eps > 0.f) || !(c->rms_eps >= 0.f)) return fail(STILL_E_INVAL, "eps must be positive");
  m->H = c->n_kv_heads;
  m->d = c->head_dim;
  m->D = c->latent_dim;
  m->d2 = 2 * m->d;
  m->nc = c->n_cross_heads;
  m->dc = c->cross_head_dim ? c->cross_head_dim : c->latent_dim;
  m->ns = c->n_self_heads;
  m->ds = c->self_head_dim ? c->self_head_dim : c->latent_dim;
  m->F = c->ffn_kind ? c->ffn_hidden : 0;
  m->Ec = m->nc * m->dc;
  m->Es = m->ns * m->ds;
  m->t = t;
  m->N = N;
  m->fp32 = c->mode == STILL_MODE_FP32;
  m->cs = m->fp32 ? 4 : 2;
  // kernel-imposed limits
  if (m->d != 64 && m->d != 128 && m->d != 256)
    return fail(STILL_E_UNSUPPORTED, "head_dim %d unsupported (64, 128 or 256)", m->d);
  if (m->dc % GEMM_BN) return fail(STILL_E_UNSUPPORTED, "cross head width %d must be a multiple of %d", m->dc, GEMM_BN);
  if (m->ns > 0 && m->ds % GEMM_BN)
    return fail(STILL_E_UNSUPPORTED, "self head width %d must be a multiple of %d", m->ds, GEMM_BN);
  if (m->D % 8) return fail(STILL_E_UNSUPPORTED, "latent_dim %d must be a multiple of 8", m->D);
  if (m->F % 8) return fail(STILL_E_UNSUPPORTED, "ffn_hidden %d must be a multiple of 8", m->F);
  // the fp16 cross-attention addresses one head's q, k and X^T with 32-bit offsets
  if ((double)N * m->nc * m->dc * 2.0 >= 4294967296.0 || (double)t * m->nc * m->dc * 2.0 >= 4294967296.0)
    return fail(STILL_E_UNSUPPORTED, "N or t too large for one head's 4 GiB key/query span");
  if (!m->fp32 && m->H > 128) return fail(STILL_E_UNSUPPORTED, "n_kv_heads %d > 128 unsupported", m->H);
  if ((long)m->H * N > (long)GEMM_BN * 65535L)
    return fail(STILL_E_UNSUPPORTED, "H*N = %lld exceeds the supported %ld rows", (long long)(m->H * N), (long)GEMM_BN * 65535L);
  m->tpad = (int)rup(t, 64);
  m->Npad = rup(N, 256);
  m->np_c = m->dc / GEMM_BN * 2;
  m->np_s = m->ns > 0 ? m->ds / GEMM_BN * 2 : 0;
  m->topk = m->fp32 ? ATT_TOPK : XATT_TOPK;
  m->ncand = m->fp32 ? 2 * ATT_TOPK : 2 * xatt_waves(m->d2) * XATT_TOPK;
  m->R = REFINE_R;
  m->att_tt = (m->fp32 || m->d2 <= 256) ? 128 : 64;
  m->splits = choose_splits(*m);
  m->keys_per_split = rup((m->N + m->splits - 1) / m->splits, key_block(*m));
  m->splits = (int)((m->N + m->keys_per_split - 1) / m->keys_per_split);
  return STILL_OK;
}

// The weight matrices of one layer in a fixed order, with their element
// counts: per block the cross-attention (if the block has it), self-attention
// and FFN matrices, then the two output heads.  `f` is called as
// f(src, elements, slot) with slot the matrix's address in a still_block_weights
// / still_layer_weights copy whose pointer is to be replaced.
template <class F>
static void for_each_matrix(const still_config* c, const Dims& m, const still_layer_weights* w,
                            still_block_weights* blocks, const void** wkey, const void** wval, F f) {
  for (int b = 0; b < c->n_blocks; ++b) {
    const still_block_weights* bw = w ? &w->blocks[b] : nullptr;
    still_block_weights* o = blocks ? &blocks[b] : nullptr;
    auto put = [&](const void* const* src, long n, const void** slot) { f(src ? *src : nullptr, n, slot); };
#define MAT(name, n) put(bw ? &bw->name : nullptr, (long)(n), o ? &o->name : nullptr)
    if (c->cross_every_block || b == 0) {
      MAT(ca_wq, (long)m.Ec * m.D);
      MAT(ca_wk, (long)m.Ec * m.d2);
      MAT(ca_wv, (long)m.Ec * m.d2);
      MAT(ca_wo, (long)m.D * m.Ec);
    }
    if (m.ns > 0) {
      MAT(sa_wq, (long)m.Es * m.D);
      MAT(sa_wk, (long)m.Es * m.D);
      MAT(sa_wv, (long)m.Es * m.D);
      MAT(sa_wo, (long)m.D * m.Es);
    }
    if (c->ffn_kind == STILL_FFN_SWIGLU) MAT(ffn_wg, (long)m.F * m.D);
    if (c->ffn_kind != STILL_FFN_NONE) {
      MAT(ffn_wu, (long)m.F * m.D);
      MAT(ffn_wd, (long)m.D * m.F);
    }
#undef MAT
  }
  f(w ? w->w_key : nullptr, (long)m.d * m.D, wkey);
  f(w ? w->w_val : nullptr, (long)m.d * m.D, wval);
}

static long matrix_elems(const still_config* c, const Dims& m) {
  long total = 0;
  for_each_matrix(c, m, nullptr, nullptr, nullptr, nullptr,
                  [&](const void*, long n, const void**) { total += rup(n, 128); });
  return total;
}

static Plan make_plan(const still_config* c, const Dims& m) {
  Plan p;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  const size_t cs = m.cs;
  const long Ht = (long)m.H * m.t;
  const long HN = (long)m.H * m.N;
  p.pq = take(sizeof(double) * m.t);
  p.tab_ck = take(8ul * m.N * (m.dc / 2));
  p.tab_cq = take(8ul * m.t * (m.dc / 2));
  p.tab_bk = take(8ul * m.N * (m.d / 2));
  p.tab_bq = take(8ul * m.t * (m.d / 2));
  p.wconv = m.fp32 ? 0 : take(2ul * matrix_elems(c, m));
  p.wkt = m.fp32 ? 0 : take(2ul * m.Ec * m.d2);
  p.X = take(cs * HN * m.d2);
  p.XT = take(cs * (size_t)m.H * m.d2 * m.Npad);
  p.Z = take(4ul * Ht * m.D);
  p.Y = take(cs * Ht * m.D);
  p.q = take(cs * Ht * m.Ec);            // also the cross-attention head outputs
  p.partq = take(4ul * Ht * m.nc * m.np_c);
  p.rq = take(4ul * Ht * m.nc);
  p.O = take(cs * Ht * m.nc * m.d2);
  if (m.R > 0) {
    const long HCT = Ht * m.nc;
    if (!m.fp32) {
      p.Ylo = take(cs * Ht * m.D);
      p.qex = take(4ul * Ht * m.Ec);
    }
    p.cval = take(4ul * m.splits * HCT * m.ncand);
    p.cidx = take(4ul * m.splits * HCT * m.ncand);
    p.ridx = take(4ul * HCT * m.R);
    p.rval = take(4ul * HCT * m.R);
    p.Xc = m.fp32 ? take(cs * HCT * m.R * 2 * m.d) : 0;   // fp16: rows gathered inside the refine kernel
    p.rpart = take(8ul * HCT * m.R * (m.fp32 ? m.dc / 64 : 1));
    p.crow = take(4ul * HCT * m.R);
    p.ccount = take(4ul * m.H * m.nc);
  }
  const size_t ubase = off;
  // k: row-major [H*N][nc*dc] (fp32 mode) or fragment-tiled with Npad keys per head (fp16)
  p.k = take(cs * (m.fp32 ? HN : (long)m.H * m.Npad) * m.Ec);
  p.partk = take(4ul * HN * m.nc * m.np_c);
  p.rk = take(4ul * HN * m.nc);
  p.opart = take(4ul * m.splits * Ht * m.nc * m.d2);
  p.mpart = take(4ul * m.splits * Ht * m.nc);
  p.lpart = take(4ul * m.splits * Ht * m.nc);
  const size_t end1 = off;
  off = ubase;
  if (m.ns > 0) {
    p.qs = take(cs * Ht * m.Es);
    p.ks = take(cs * Ht * m.Es);
    p.vT = take(cs * (size_t)m.H * m.Es * m.tpad);
    p.partqs = take(4ul * Ht * m.ns * m.np_s);
    p.partks = take(4ul * Ht * m.ns * m.np_s);
    p.rqs = take(4ul * Ht * m.ns);
    p.rks = take(4ul * Ht * m.ns);
    p.Ssa = take(4ul * (size_t)m.H * m.ns * m.t * m.tpad);
    p.Psa = take(cs * (size_t)m.H * m.ns * m.t * m.tpad);
    p.Osa = take(cs * Ht * m.Es);
  }
  p.hid = take(cs * Ht * (m.F > 0 ? m.F : 1));
  p.total = (off > end1 ? off : end1) + 256;
  return p;
}

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

// WIDE: 128 x 256 tiles (BK 32, 2 waves per SIMD) for the latent-side
// products with many output columns and K >= 512 (fp16 mode; paired kinds need
// head widths that are multiples of 256), where they still leave at least two
// workgroups per CU.  The norm partials of a PAIR product then number hd/256*2
// per head instead of hd/128*2, so paired kinds always take them.
template <class CT, class TA, class TB, class TC, class TBias, int EPI, bool WIDE = false>
static hipError_t gemm(const GemmArgs& g, int batch, hipStream_t st, int cls = STILL_K_LATENT) {
  timing::Scope ts(cls, st);
  if constexpr (WIDE && sizeof(CT) == 2) {
    constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU || EPI == EPI_REFINE);
    const long ntn = PAIRED ? (g.N + 127) / 128 : (g.N + 255) / 256;
    const long ntm = g.mgroups > 1 ? (g.M / g.mgroups + 128 / g.mgroups - 1) / (128 / g.mgroups) : (g.M + 127) / 128;
    if (PAIRED || ntn * ntm * batch >= 512) return launch_gemm<CT, TA, TB, TC, TBias, EPI, 128, 256, 32>(g, batch, st);
  }
  if constexpr (sizeof(CT) == 2 && EPI != EPI_REFINE) {
    // fewer 128-row tiles than CUs (the output heads, small t): 64-row tiles
    constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU);
    const long ntn = PAIRED ? (g.N + 63) / 64 : (g.N + 127) / 128;
    const long ntm = g.mgroups > 1 ? (g.M / g.mgroups + 128 / g.mgroups - 1) / (128 / g.mgroups) : (g.M + 127) / 128;
    if (g.mgroups <= 1 && ntn * ntm * batch < 256) {
      if (g.K >= GEMM_LONG_K)
        return launch_gemm<CT, TA, TB, TC, TBias, EPI, 64, Tile<CT>::BN, 2 * Tile<CT>::BK>(g, batch, st);
      return launch_gemm<CT, TA, TB, TC, TBias, EPI, 64, Tile<CT>::BN, Tile<CT>::BK>(g, batch, st);
    }
  }
  if (g.K >= GEMM_LONG_K)
    return launch_gemm<CT, TA, TB, TC, TBias, EPI, Tile<CT>::BM, Tile<CT>::BN, 2 * Tile<CT>::BK>(g, batch, st);
  return launch_gemm<CT, TA, TB, TC, TBias, EPI, Tile<CT>::BM, Tile<CT>::BN, Tile<CT>::BK>(g, batch, st);
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

static inline int grid1d(long n, int per = 256) {
  long b = (n + per - 1) / per;
  if (b > 65535L * 16) b = 65535L * 16;
  if (b < 1) b = 1;
  return (int)b;
}

template <class CT, int D2>
static hipError_t launch_attn(const AttnArgs& a, int splits, hipStream_t st) {
  dim3 grid((a.t + ATT_TT - 1) / ATT_TT, a.H * a.nc, splits);
  if constexpr (sizeof(CT) == 2) {
    constexpr int TT = D2 <= 256 ? 128 : 64;
    const int ntt = (a.t + TT - 1) / TT;
    static_assert(xatt_waves(D2) == 4, "the fp16 kernel runs 4 waves");
    hipLaunchKernelGGL((xattn_f16_kernel<TT, D2, XATT_TOPK>), dim3(ntt * a.H * a.nc * splits), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((cross_attn_kernel<CT, ATT_TT, (D2 > 256 ? 32 : ATT_NB), 32, D2, ATT_TOPK>), grid, dim3(256),
                       0, st, a);
  }
  return hipGetLastError();
}

// per-call tables shared by all layers
static still_status prepare_tables(const Dims& m, const Plan& p, char* ws, const double* positions,
                                   double rope_theta, double cbase, bool rerotate, double* out_positions,
                                   hipStream_t st) {
  double* pq = (double*)(ws + p.pq);
  TIMED(STILL_K_OTHER);
  hipLaunchKernelGGL(positions_kernel, dim3(1), dim3(256), 0, st, positions, m.N, m.t, pq, out_positions);
  HIP_TRY(hipGetLastError());
  auto table = [&](const double* pos, long R, int w, double base, size_t off) -> hipError_t {
    hipLaunchKernelGGL(rope_table_kernel, dim3(grid1d(R * (w / 2))), dim3(256), 0, st, pos, R, w, base,
                       (float2*)(ws + off));
    return hipGetLastError();
  };
  HIP_TRY(table(positions, m.N, m.dc, cbase, p.tab_ck));
  HIP_TRY(table(pq, m.t, m.dc, cbase, p.tab_cq));
  HIP_TRY(table(positions, m.N, m.d, rope_theta, p.tab_bk));
  if (rerotate) HIP_TRY(table(pq, m.t, m.d, rope_theta, p.tab_bq));
  return STILL_OK;
}

// ---------------------------------------------------------------------------
// One layer: IT = I/O type of K, V, weights and outputs; CT = MFMA operand /
// intermediate storage type.
// ---------------------------------------------------------------------------
template <class IT, class CT>
static still_status run_layer(const still_config* cfg, const Dims& m, const Plan& p, char* ws,
                              const still_layer_weights* w, const void* Kp, const void* Vp, bool rerotate,
                              void* Ckp, void* Cvp, hipStream_t st) {
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
  const float2* tab_ck = (const float2*)(ws + p.tab_ck);
  const float2* tab_cq = (const float2*)(ws + p.tab_cq);
  const float2* tab_bk = (const float2*)(ws + p.tab_bk);
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

  // RoPE-fix staging of X = [R(-p) K ; V] and X^T
  {
    int RW = 64;
    while (RW > 8 && (size_t)RW * (m.d2 + 8) * m.cs > 40960) RW /= 2;
    const size_t lds = (size_t)RW * (m.d2 + 8) * m.cs;
    dim3 grid((unsigned)((m.Npad + RW - 1) / RW), m.H);
    TIMED(STILL_K_OTHER);
    hipLaunchKernelGGL((stage_x_kernel<IT, CT>), grid, dim3(256), lds, st, (const IT*)Kp, (const IT*)Vp, tab_bk, m.N,
                       m.d, X, XT, m.Npad, RW);
    HIP_TRY(hipGetLastError());
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
        ka.tab = tab_ck;
        ka.k = (f16*)k;
        ka.part = partk;
        ka.H = m.H;
        ka.N = (int)m.N;
        ka.nc = m.nc;
        ka.dc = m.dc;
        ka.npad = m.Npad;
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
          constexpr bool SPLIT = sizeof(CT) == 2;   // fp16: [K_hi | V | K_lo], fp32: [K | V]
          const int W = SPLIT ? 3 * m.d : 2 * m.d;
          const long HCT = Ht * m.nc;
          int* ridx = (int*)(ws + p.ridx);
          {
            TIMED(STILL_K_REFINE);
            hipLaunchKernelGGL(refine_select_kernel, dim3((unsigned)((HCT + 255) / 256)), dim3(256), 0, st, a.cval,
                               a.cidx, a.mpart, m.splits, HCT, m.ncand, m.R, ridx, (float*)(ws + p.rval));
            HIP_TRY(hipGetLastError());
            const int TR = m.t * m.R, NB = m.H * m.nc;
            int* crow = (int*)(ws + p.crow);
            int* ccount = (int*)(ws + p.ccount);
            hipLaunchKernelGGL(refine_compact_kernel, dim3(NB), dim3(256), 0, st, ridx, TR, crow, ccount);
            HIP_TRY(hipGetLastError());
            if constexpr (SPLIT) {   // fp16: gather, exact key projection and dot product in one kernel
              RefineKArgs rk_;
              rk_.K = Kp;
              rk_.V = Vp;
              rk_.tab_b = tab_bk;
              rk_.tab_c = tab_ck;
              rk_.wkt = (const f16*)(ws + p.wkt);
              rk_.bias = bw.ca_bk;
              rk_.ridx = ridx;
              rk_.crow = crow;
              rk_.count = ccount;
              rk_.qex = (const float*)(ws + p.qex);
              rk_.rpart = (float2*)(ws + p.rpart);
              rk_.N = m.N;
              rk_.t = m.t;
              rk_.R = m.R;
              rk_.nc = m.nc;
              rk_.dc = m.dc;
              constexpr int BMR = 64;   // candidate rows per workgroup (LDS: BMR x 3d fp16; 2-3 workgroups per CU)
              rk_.H = m.H;
              rk_.ntile = (TR + BMR - 1) / BMR;
              const dim3 rg((unsigned)(rk_.ntile * NB));
              if (m.d == 64) hipLaunchKernelGGL((refine_kernel<64, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              else if (m.d == 128) hipLaunchKernelGGL((refine_kernel<128, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              else hipLaunchKernelGGL((refine_kernel<256, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              HIP_TRY(hipGetLastError());
            } else {
              hipLaunchKernelGGL((refine_gather_kernel<IT, CT>), dim3(grid1d(HCT * m.R * (m.d / 2))), dim3(256), 0,
                                 st, (const IT*)Kp, (const IT*)Vp, tab_bk, ridx, crow, ccount, m.N, m.d, m.nc, TR, NB,
                                 (CT*)(ws + p.Xc));
              HIP_TRY(hipGetLastError());
            }
          }
          if constexpr (!SPLIT) {  // fp32: exact k~ of the packed keys [K | V] [W_K]^T, dotted with q~
            GemmArgs g = gargs(m.t * m.R, m.dc / 2, W, ws + p.Xc, W, bw.ca_wk, m.d2, nullptr, 0);
            g.nb2 = m.nc;
            g.sA1 = (long)m.nc * m.t * m.R * W;
            g.sA2 = (long)m.t * m.R * W;
            g.sB2 = (long)m.dc * m.d2;
            g.bwrap = 0;
            g.bias = bw.ca_bk;
            g.sBias2 = m.dc;
            g.hd = m.dc;
            g.tab = tab_ck;
            g.ridx = ridx;
            g.crow = (const int*)(ws + p.crow);
            g.mcount = (const int*)(ws + p.ccount);
            g.sI1 = (long)m.nc * m.t * m.R;
            g.sI2 = (long)m.t * m.R;
            g.R = m.R;
            g.qex = (const float*)q;   // fp32 mode: q is exact fp32
            g.ldqex = m.Ec;
            g.sE1 = (long)m.t * m.Ec;
            g.sE2 = m.dc;
            g.rpart = (float2*)(ws + p.rpart);
            g.sR1 = (long)m.nc * m.t * m.R * (m.dc / 64);
            g.sR2 = (long)m.t * m.R * (m.dc / 64);
            HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_REFINE>(g, m.H * m.nc, st, STILL_K_REFINE)));
          }
          ra.R = m.R;
          ra.NP = SPLIT ? 1 : m.dc / 64;
          ra.ridx = ridx;
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
      {  // Z += Concat(heads) W_O^T
        GemmArgs g = gargs((int)Ht, m.D, m.Ec, head, m.Ec, bw.ca_wo, m.Ec, Z, m.D);
        HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_RESID, true>(g, 1, st)));
      }
    }
    // ---------------- latent self-attention: Z += SelfAttn(RMSNorm(Z))
    if (m.ns > 0) {
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

// ---------------------------------------------------------------------------
// Validation of a layer's pointers
// ---------------------------------------------------------------------------
static bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

static still_status check_ptr(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(STILL_E_INVAL, "%s is NULL", name) : STILL_OK;
  if (misaligned(p)) return fail(STILL_E_INVAL, "%s is not 16-byte aligned", name);
  return STILL_OK;
}

static still_status check_layer(const still_config* c, const Dims& m, const still_layer_weights* w, int layer) {
  if (!w) return fail(STILL_E_INVAL, "layer %d: weights NULL", layer);
  if (w->t_bank != m.t) return fail(STILL_E_SHAPE, "layer %d: t=%d but latent bank holds %d", layer, m.t, w->t_bank);
  still_status s;
#define CHK(p, req)                                                        \
  if ((s = check_ptr((p), #p, (req))) != STILL_OK) {                       \
    g_last_error = "layer " + std::to_string(layer) + ": " + g_last_error; \
    return s;                                                              \
  }
  CHK(w->latents, true);
  CHK(w->w_key, true);
  CHK(w->w_val, true);
  if (!w->blocks) return fail(STILL_E_INVAL, "layer %d: blocks NULL", layer);
  for (int b = 0; b < c->n_blocks; ++b) {
    const still_block_weights& bw = w->blocks[b];
    const bool ca = c->cross_every_block || b == 0;
    CHK(bw.ca_wq, ca);
    CHK(bw.ca_bq, false);
    CHK(bw.ca_wk, ca);
    CHK(bw.ca_bk, false);
    CHK(bw.ca_wv, ca);
    CHK(bw.ca_wo, ca);
    const bool sa = m.ns > 0;
    CHK(bw.sa_wq, sa);
    CHK(bw.sa_bq, false);
    CHK(bw.sa_wk, sa);
    CHK(bw.sa_bk, false);
    CHK(bw.sa_wv, sa);
    CHK(bw.sa_wo, sa);
    CHK(bw.ffn_wg, c->ffn_kind == STILL_FFN_SWIGLU);
    CHK(bw.ffn_wu, c->ffn_kind != STILL_FFN_NONE);
    CHK(bw.ffn_wd, c->ffn_kind != STILL_FFN_NONE);
  }
#undef CHK
  return STILL_OK;
}

static still_status compact(const still_config* cfg, int32_t L, const still_layer_weights* w, const void* const* K,
                            const void* const* V, const double* positions, int64_t N, double rope_theta, int32_t t,
                            uint32_t flags, void* const* Ck, void* const* Cv, double* out_positions,
                            const void* const* w_beta, const still_beta_opts* bopt, float* const* beta,
                            void* workspace, size_t workspace_bytes, void* stream) {
  Dims m;
  still_status s = make_dims(cfg, N, t, &m);
  if (s != STILL_OK) return s;
  if (L < 1) return fail(STILL_E_INVAL, "n_layers must be >= 1");
  if (!w || !K || !V || !Ck || !Cv) return fail(STILL_E_INVAL, "NULL layer array");
  if (flags & ~(uint32_t)STILL_F_REROTATE) return fail(STILL_E_INVAL, "unknown flags 0x%x", flags);
  if (!(rope_theta > 0.0)) return fail(STILL_E_INVAL, "rope_theta must be > 0");
  if (!positions) return fail(STILL_E_INVAL, "positions is NULL");
  if (((uintptr_t)positions & 7u) || ((uintptr_t)out_positions & 7u))
    return fail(STILL_E_INVAL, "positions / out_positions must be 8-byte aligned");
  for (int l = 0; l < L; ++l) {
    if ((s = check_layer(cfg, m, &w[l], l)) != STILL_OK) return s;
    if (!K[l] || !V[l] || !Ck[l] || !Cv[l]) return fail(STILL_E_INVAL, "layer %d: NULL cache or output pointer", l);
    if (misaligned(K[l]) || misaligned(V[l]) || misaligned(Ck[l]) || misaligned(Cv[l]))
      return fail(STILL_E_INVAL, "layer %d: cache/output pointers must be 16-byte aligned", l);
  }
  BetaShape shape{0.f, 0.f};
  if (beta) {
    if (!w_beta) return fail(STILL_E_INVAL, "beta outputs given without w_beta");
    for (int l = 0; l < L; ++l)
      if (!w_beta[l] || !beta[l] || ((uintptr_t)beta[l] & 3u) || ((uintptr_t)w_beta[l] & (m.fp32 ? 3u : 1u)))
        return fail(STILL_E_INVAL, "layer %d: NULL or misaligned w_beta / beta", l);
    if (bopt) {
      if (!std::isfinite(bopt->beta_max) || !std::isfinite(bopt->mass_alpha) || !std::isfinite(bopt->log_x))
        return fail(STILL_E_INVAL, "beta options must be finite");
      shape.beta_max = bopt->beta_max > 0.f ? bopt->beta_max : 0.f;
      shape.offset = (float)(bopt->mass_alpha * std::log((double)N / (double)t) + bopt->log_x);
    }
  }
  const Plan p = make_plan(cfg, m);
  if (!workspace) return fail(STILL_E_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < p.total)
    return fail(STILL_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, p.total);
  char* ws = (char*)(((uintptr_t)workspace + 255) & ~(uintptr_t)255);
  hipStream_t st = (hipStream_t)stream;
  (void)hipGetLastError();  // clear a stale error so launch checks report this call
  const bool rerot = (flags & STILL_F_REROTATE) != 0;
  if ((s = prepare_tables(m, p, ws, positions, rope_theta, cfg->compactor_rope_base, rerot, out_positions, st)) !=
      STILL_OK)
    return s;
  for (int l = 0; l < L; ++l) {
    s = m.fp32 ? run_layer<float, float>(cfg, m, p, ws, &w[l], K[l], V[l], rerot, Ck[l], Cv[l], st)
               : run_layer<bf16, f16>(cfg, m, p, ws, &w[l], K[l], V[l], rerot, Ck[l], Cv[l], st);
    if (s != STILL_OK) return s;
    if (beta) {  // beta = shape(Z_out w_beta) from the final latent state left in the workspace
      TIMED(STILL_K_OTHER);
      const long rows = (long)m.H * m.t;
      const float* Z = (const float*)(ws + p.Z);
      if (m.fp32)
        hipLaunchKernelGGL((beta_kernel<float>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, Z,
                           (const float*)w_beta[l], rows, m.D, cfg->final_norm, cfg->rms_eps, shape, beta[l]);
      else
        hipLaunchKernelGGL((beta_kernel<bf16>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, Z,
                           (const bf16*)w_beta[l], rows, m.D, cfg->final_norm, cfg->rms_eps, shape, beta[l]);
      if (hipGetLastError() != hipSuccess) return fail(STILL_E_HIP, "beta launch failed");
    }
  }
  return STILL_OK;
}

// ---------------------------------------------------------------------------
// Consumer attention over [C_k; K] with bias [beta; 0]
// ---------------------------------------------------------------------------
struct AttendPlan {
  int R, splits, cps, kc;
  size_t opart, mpart, lpart, total;
};

constexpr int ATTEND_TARGET_BLOCKS = 2048;   // one-wave blocks per launch that keep the chip streaming

static still_status attend_plan(const still_attend_config* c, AttendPlan* ap) {
  if (!c) return fail(STILL_E_INVAL, "attend config is NULL");
  if (c->mode != STILL_MODE_BF16 && c->mode != STILL_MODE_FP32) return fail(STILL_E_DTYPE, "unknown mode %d", c->mode);
  if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256)
    return fail(STILL_E_UNSUPPORTED, "attend head_dim %d not in {64, 128, 256}", c->head_dim);
  if (c->n_kv_heads < 1 || c->group < 1 || c->n_queries < 1) return fail(STILL_E_SHAPE, "attend sizes must be >= 1");
  if ((long)c->group * c->n_queries > ATTEND_MAX_ROWS)
    return fail(STILL_E_UNSUPPORTED, "group * n_queries = %ld exceeds %d", (long)c->group * c->n_queries,
                ATTEND_MAX_ROWS);
  if (c->n_kv_heads > 65535) return fail(STILL_E_UNSUPPORTED, "n_kv_heads above 65535");
  if (c->t < 0 || c->n_suffix < 0 || (long)c->t + c->n_suffix < 1 || (long)c->t + c->n_suffix > (1L << 30))
    return fail(STILL_E_SHAPE, "attend needs 1 <= t + n_suffix <= 2^30 (t=%d, n_suffix=%d)", c->t, c->n_suffix);
  if (c->causal != 0 && c->causal != 1) return fail(STILL_E_INVAL, "causal must be 0 or 1");
  if (c->causal && c->n_suffix < c->n_queries)
    return fail(STILL_E_SHAPE, "causal attention needs n_suffix >= n_queries");
  if (!std::isfinite(c->scale) || c->scale < 0.f) return fail(STILL_E_INVAL, "scale must be finite and >= 0");
  if (!(c->rope_theta >= 0.0) || !std::isfinite(c->rope_theta)) return fail(STILL_E_INVAL, "rope_theta must be >= 0");
  // keys per chunk: the decode kernel's KC (rows <= 8) or the LDS kernel's 64
  const long R = (long)c->group * c->n_queries;
  const int esize = c->mode == STILL_MODE_FP32 ? 4 : 2;
  const int kc = R <= ATTEND_DECODE_ROWS ? (R <= 4 ? 8 : 4) * (64 / (c->head_dim * esize / 16)) : ATTEND_KC;
  ap->kc = kc;
  const long chunks = ((long)c->t + kc - 1) / kc + ((long)c->n_suffix + kc - 1) / kc;
  const long per_head = std::max(1L, (long)ATTEND_TARGET_BLOCKS / c->n_kv_heads);
  ap->R = c->group * c->n_queries;
  ap->cps = (int)((chunks + per_head - 1) / per_head);
  ap->splits = (int)((chunks + ap->cps - 1) / ap->cps);
  const size_t slots = (size_t)ap->splits * c->n_kv_heads * ap->R;
  ap->opart = 0;
  ap->mpart = rup((long)(slots * c->head_dim * sizeof(float)), 256);
  ap->lpart = ap->mpart + rup((long)(slots * sizeof(float)), 256);
  ap->total = ap->lpart + rup((long)(slots * sizeof(float)), 256) + 256;   // + alignment slack
  return STILL_OK;
}

template <class IT, int D>
static hipError_t launch_attend(const ConsumerArgs& a, hipStream_t st) {
  const int R = a.group * a.nq;
  const dim3 grid(a.splits, a.H);
  if (R <= 2)
    hipLaunchKernelGGL((attend_decode_kernel<IT, D, 2>), grid, dim3(64), 0, st, a);
  else if (R <= 4)
    hipLaunchKernelGGL((attend_decode_kernel<IT, D, 4>), grid, dim3(64), 0, st, a);
  else if (R <= ATTEND_DECODE_ROWS)
    hipLaunchKernelGGL((attend_decode_kernel<IT, D, 8>), grid, dim3(64), 0, st, a);
  else if (R <= 16)
    hipLaunchKernelGGL((attend_partial_kernel<IT, D, 16>), grid, dim3(64), (attend_lds_bytes<IT, D>(16)), st, a);
  else
    hipLaunchKernelGGL((attend_partial_kernel<IT, D, ATTEND_MAX_ROWS>), grid, dim3(64),
                       (attend_lds_bytes<IT, D>(ATTEND_MAX_ROWS)), st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attend_merge_kernel<IT, D>), dim3(a.group * a.nq, a.H), dim3(64 * ATTEND_MERGE_WAVES), 0,
                     st, a);
  return hipGetLastError();
}

}  // namespace still

using namespace still;

extern "C" {

size_t still_workspace_size(const still_config* cfg, int64_t N, int32_t t, int32_t n_layers) {
  Dims m;
  if (n_layers < 1 || make_dims(cfg, N, t, &m) != STILL_OK) return 0;
  return make_plan(cfg, m).total;
}

still_status still_compact_layer(const still_config* cfg, const still_layer_weights* w, const void* K, const void* V,
                                 const double* positions, int64_t N, double rope_theta, int32_t t, uint32_t flags,
                                 void* C_k, void* C_v, double* out_positions, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  const void* Ka[1] = {K};
  const void* Va[1] = {V};
  void* Cka[1] = {C_k};
  void* Cva[1] = {C_v};
  return compact(cfg, 1, w, Ka, Va, positions, N, rope_theta, t, flags, Cka, Cva, out_positions, nullptr, nullptr,
                 nullptr, workspace, workspace_bytes, stream);
}

still_status still_compact_model(const still_config* cfg, int32_t n_layers, const still_layer_weights* w,
                                 const void* const* K, const void* const* V, const double* positions, int64_t N,
                                 double rope_theta, int32_t t, uint32_t flags, void* const* C_k, void* const* C_v,
                                 double* out_positions, void* workspace, size_t workspace_bytes, void* stream) {
  return compact(cfg, n_layers, w, K, V, positions, N, rope_theta, t, flags, C_k, C_v, out_positions, nullptr,
                 nullptr, nullptr, workspace, workspace_bytes, stream);
}

still_status still_compact_model_beta(const still_config* cfg, int32_t n_layers, const still_layer_weights* w,
                                      const void* const* K, const void* const* V, const double* positions, int64_t N,
                                      double rope_theta, int32_t t, uint32_t flags, void* const* C_k,
                                      void* const* C_v, double* out_positions, const void* const* w_beta,
                                      const still_beta_opts* beta_opts, float* const* beta, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (!beta) return fail(STILL_E_INVAL, "beta output array is NULL");
  return compact(cfg, n_layers, w, K, V, positions, N, rope_theta, t, flags, C_k, C_v, out_positions, w_beta,
                 beta_opts, beta, workspace, workspace_bytes, stream);
}

size_t still_attend_workspace_size(const still_attend_config* cfg) {
  AttendPlan ap;
  const std::string keep = g_last_error;
  if (attend_plan(cfg, &ap) != STILL_OK) {
    g_last_error = keep;
    return 0;
  }
  return ap.total;
}

still_status still_attend(const still_attend_config* cfg, const void* q, const double* q_positions,
                          const void* C_k, const void* C_v, const float* beta, const void* K, const void* V,
                          void* out, void* workspace, size_t workspace_bytes, void* stream) {
  AttendPlan ap;
  still_status s = attend_plan(cfg, &ap);
  if (s != STILL_OK) return s;
  if ((s = check_ptr(q, "q", true)) != STILL_OK || (s = check_ptr(out, "out", true)) != STILL_OK ||
      (s = check_ptr(C_k, "C_k", cfg->t > 0)) != STILL_OK || (s = check_ptr(C_v, "C_v", cfg->t > 0)) != STILL_OK ||
      (s = check_ptr(K, "K", cfg->n_suffix > 0)) != STILL_OK || (s = check_ptr(V, "V", cfg->n_suffix > 0)) != STILL_OK)
    return s;
  if (beta && ((uintptr_t)beta & 3u)) return fail(STILL_E_INVAL, "beta is not 4-byte aligned");
  if (cfg->rope_theta > 0.0 && (!q_positions || ((uintptr_t)q_positions & 7u)))
    return fail(STILL_E_INVAL, "rope_theta > 0 needs 8-byte aligned q_positions");
  if (!workspace) return fail(STILL_E_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < ap.total)
    return fail(STILL_E_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, ap.total);
  char* ws = (char*)(((uintptr_t)workspace + 255) & ~(uintptr_t)255);
  ConsumerArgs a;
  a.q = q;
  a.ck = C_k;
  a.cv = C_v;
  a.beta = cfg->t > 0 ? beta : nullptr;
  a.k = K;
  a.v = V;
  a.out = out;
  a.opart = (float*)(ws + ap.opart);
  a.mpart = (float*)(ws + ap.mpart);
  a.lpart = (float*)(ws + ap.lpart);
  a.H = cfg->n_kv_heads;
  a.group = cfg->group;
  a.nq = cfg->n_queries;
  a.t = cfg->t;
  a.S = cfg->n_suffix;
  a.causal = cfg->causal;
  a.splits = ap.splits;
  a.cps = ap.cps;
  a.qpos = cfg->rope_theta > 0.0 ? q_positions : nullptr;
  a.theta = cfg->rope_theta;
  a.scale = cfg->scale != 0.f ? cfg->scale : 1.f / std::sqrt((float)cfg->head_dim);
  hipStream_t st = (hipStream_t)stream;
  (void)hipGetLastError();
  hipError_t e;
  {
    TIMED(STILL_K_ATTEND);
    const bool f32 = cfg->mode == STILL_MODE_FP32;
    switch (cfg->head_dim) {
      case 64: e = f32 ? launch_attend<float, 64>(a, st) : launch_attend<bf16, 64>(a, st); break;
      case 128: e = f32 ? launch_attend<float, 128>(a, st) : launch_attend<bf16, 128>(a, st); break;
      default: e = f32 ? launch_attend<float, 256>(a, st) : launch_attend<bf16, 256>(a, st); break;
    }
  }
  if (e != hipSuccess) return fail(STILL_E_HIP, "attend launch: %s", hipGetErrorString(e));
  return STILL_OK;
}

const char* still_status_string(int32_t s) {
  switch (s) {
    case STILL_OK: return "STILL_OK";
    case STILL_E_INVAL: return "STILL_E_INVAL";
    case STILL_E_SHAPE: return "STILL_E_SHAPE";
    case STILL_E_DTYPE: return "STILL_E_DTYPE";
    case STILL_E_WORKSPACE: return "STILL_E_WORKSPACE";
    case STILL_E_UNSUPPORTED: return "STILL_E_UNSUPPORTED";
    case STILL_E_HIP: return "STILL_E_HIP";
    default: return "STILL_E_UNKNOWN";
  }
}

const char* still_last_error(void) { return g_last_error.c_str(); }

const char* still_version(void) { return "still-mi355x 0.1 (gfx950)"; }

still_status still_timing_enable(int32_t class_mask) {
  timing::mask = (unsigned)class_mask & ((1u << STILL_K_COUNT) - 1u);
  return STILL_OK;
}

still_status still_timing_reset(void) {
  hipError_t e = timing::harvest(timing::pending.size());
  for (int i = 0; i < STILL_K_COUNT; ++i) {
    timing::ms[i] = 0.0;
    timing::count[i] = 0;
  }
  if (e != hipSuccess) return fail(STILL_E_HIP, "timing reset: %s", hipGetErrorString(e));
  return STILL_OK;
}

still_status still_timing_read(int32_t cls, double* total_ms, int64_t* launches) {
  if (cls < 0 || cls >= STILL_K_COUNT || !total_ms || !launches) return fail(STILL_E_INVAL, "bad timing query");
  hipError_t e = timing::harvest(timing::pending.size());
  if (e != hipSuccess) return fail(STILL_E_HIP, "timing read: %s", hipGetErrorString(e));
  *total_ms = timing::ms[cls];
  *launches = timing::count[cls];
  return STILL_OK;
}

}  // extern "C"
