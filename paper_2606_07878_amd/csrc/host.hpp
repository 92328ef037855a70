// host.hpp - host-side plumbing shared by the library's translation units:
// error reporting, optional kernel timing, the derived dimensions of a call
// and its workspace plan.
#pragma once
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
#include "misc.hpp"

namespace still {

inline thread_local std::string g_last_error;

inline still_status fail(still_status s, const char* fmt, ...) {
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

inline long rup(long x, long m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------------------
// Optional per-class kernel timing with hipEvent pairs on the launch stream.
// ---------------------------------------------------------------------------
namespace timing {
struct Rec {
  int cls;
  hipEvent_t a, b;
};
inline unsigned mask = 0;   // bit c: record launches of class c
inline std::vector<Rec> pending;
inline std::vector<hipEvent_t> spare;
inline double ms[STILL_K_COUNT];
inline long long count[STILL_K_COUNT];

inline hipEvent_t get_event() {
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
inline hipError_t harvest(size_t n) {
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
// keys per latent whose logits are recomputed accurately: every candidate
// within the refinement margin, up to this many
constexpr int REFINE_R = 256;
static_assert(REFINE_R <= REFINE_RMAX, "merge_kernel handles up to REFINE_RMAX refined keys per latent");
// refinement rows per list the fp16 refinement grid covers at once (its
// workgroups loop over further tiles): about 4 per latent
constexpr int REFINE_GRID_R = 4;
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
  int ncand;            // candidate slots per (split, latent row) written by the attention kernel
  int ncand_fixed;      // ... of which the fixed lists (then up to ATT_OVF / XATT_OVF overflow entries)
  int att_tt;           // latents per attention workgroup
  int splits;           // split-N factor of the cross-attention
  long keys_per_split;
  // latent self-attention on the fp16 flash kernel (bf16 mode, d_s of 128,
  // 256 or 512): keys and values in its tiled layouts with tpadk keys per
  // head, split over sa_splits key ranges; otherwise scores, softmax and
  // product as separate passes
  bool sa_flash;
  int tpadk, sa_splits;
  long sa_kps;
  size_t cs;            // bytes of the compute/storage type
  bool fp32;
};

struct Plan {
  size_t pq, tab_ck, tab_cq, tab_bq;   // (cos, sin) tables of the latent positions (and, fp32 mode, of the keys)
  size_t wconv;          // bf16 mode: the layer's weight matrices converted to fp16
  size_t wkt;            // bf16 mode: fragment-tiled fp16 copy of the cross-attention W_K
  size_t X, XT, Z, Y, q, partq, rq, O;
  size_t Ylo, qex, cval, cidx, ocnt, ridx, rval, rcnt, rpart, crow, ccount;   // logit refinement
  size_t q64;                   // fp32 mode: fp64 queries of the refinement
  size_t invf_b, invf_c;        // fp64 RoPE frequencies (base, compactor)
  size_t kvpart, hscale;        // bf16 mode: per-head fp16 range scale of the staged cache
  // union region: cross-attention key side ...
  size_t k, partk, rk, opart, mpart, lpart;
  // ... or self-attention / FFN buffers
  size_t qs, ks, vT, partqs, partks, rqs, rks, Ssa, Psa, Osa, hid;
  size_t opart_s, mpart_s, lpart_s;   // flash self-attention partials
  size_t total;
};

inline int key_block(const Dims& m) { return m.fp32 ? ATT_NB : XATT_KB; }

inline int choose_splits(const Dims& m) {
  const long wgs = (long)((m.t + m.att_tt - 1) / m.att_tt) * m.H * m.nc;
  const long nblocks = (m.N + key_block(m) - 1) / key_block(m);
  // fp16 kernel: one workgroup per CU, aim for >= 2 per CU; fp32: >= 4
  long s = ((m.fp32 ? 1024 : 512) + wgs - 1) / wgs;
  if (s > nblocks) s = nblocks;
  if (s < 1) s = 1;
  return (int)s;
}

inline still_status make_dims(const still_config* c, int64_t N, int32_t t, Dims* m) {
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
  m->ncand_fixed = m->fp32 ? 2 * ATT_TOPK : 2 * xatt_waves(m->d2) * XATT_TOPK;
  m->ncand = m->ncand_fixed + (m->fp32 ? ATT_OVF : XATT_OVF);
  m->R = REFINE_R;
  m->att_tt = (m->fp32 || m->d2 <= 256) ? 128 : 64;
  m->splits = choose_splits(*m);
  m->keys_per_split = rup((m->N + m->splits - 1) / m->splits, key_block(*m));
  m->splits = (int)((m->N + m->keys_per_split - 1) / m->keys_per_split);
  m->tpadk = (int)rup(t, XATT_KB);
  m->sa_flash = !m->fp32 && m->ns > 0 && (m->ds == 128 || m->ds == 256 || m->ds == 512) &&
                (double)m->tpadk * m->Es * 2.0 < 4294967296.0;
  m->sa_splits = 1;
  m->sa_kps = m->tpadk;
  if (m->sa_flash) {
    const int tt = m->ds <= 256 ? 128 : 64;
    const long wgs = (long)((t + tt - 1) / tt) * m->H * m->ns;
    long s = (512 + wgs - 1) / wgs;
    if (s > m->tpadk / XATT_KB) s = m->tpadk / XATT_KB;
    if (s < 1) s = 1;
    m->sa_kps = rup((t + s - 1) / s, XATT_KB);
    m->sa_splits = (int)((t + m->sa_kps - 1) / m->sa_kps);
  }
  return STILL_OK;
}

// The weight matrices of one layer in a fixed order, with their element
// counts: per block the cross-attention (if the block has it), self-attention
// and FFN matrices, then the two output heads.  `f` is called as
// f(src, elements, slot) with slot the matrix's address in a still_block_weights
// / still_layer_weights copy whose pointer is to be replaced.
template <class F>
inline void for_each_matrix(const still_config* c, const Dims& m, const still_layer_weights* w,
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

inline long matrix_elems(const still_config* c, const Dims& m) {
  long total = 0;
  for_each_matrix(c, m, nullptr, nullptr, nullptr, nullptr,
                  [&](const void*, long n, const void**) { total += rup(n, 128); });
  return total;
}

// Cache rows per workgroup of the RoPE-fix staging kernel (its LDS tile of
// rows x (2d + 8) elements stays within 40 KB) and its workgroups per head.
inline int stage_rows(const Dims& m) {
  int RW = 64;
  while (RW > 8 && (size_t)RW * (m.d2 + 8) * m.cs > 40960) RW /= 2;
  return RW;
}
inline int stage_blocks(const Dims& m) { return (int)((m.Npad + stage_rows(m) - 1) / stage_rows(m)); }

inline Plan make_plan(const still_config* c, const Dims& m) {
  Plan p = {};
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
  // compactor-RoPE table of the keys: fp32 mode only (bf16 mode: rotations
  // computed in place from the positions and the fp64 frequencies)
  p.tab_ck = m.fp32 ? take(8ul * m.N * (m.dc / 2)) : 0;
  p.invf_c = take(8ul * (m.dc / 2));
  p.tab_cq = take(8ul * m.t * (m.dc / 2));
  p.invf_b = take(8ul * (m.d / 2));   // base RoPE frequencies (fp64): staging and refinement rotate in place
  p.tab_bq = take(8ul * m.t * (m.d / 2));
  p.wconv = m.fp32 ? 0 : take(2ul * matrix_elems(c, m));
  p.kvpart = m.fp32 ? 0 : take(4ul * m.H * stage_blocks(m));
  p.hscale = m.fp32 ? 0 : take(4ul * 2 * m.H);
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
    p.ocnt = take(4ul * m.splits * HCT);
    p.ridx = take(4ul * HCT * m.R);
    p.rval = take(4ul * HCT * m.R);
    p.rcnt = take(4ul * HCT);
    p.rpart = take(8ul * HCT * m.R);
    if (m.fp32) {
      p.q64 = take(8ul * Ht * m.Ec);
    }
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
    p.partqs = take(4ul * Ht * m.ns * m.np_s);
    p.partks = take(4ul * Ht * m.ns * m.np_s);
    p.rqs = take(4ul * Ht * m.ns);
    p.rks = take(4ul * Ht * m.ns);
    p.Osa = take(cs * Ht * m.Es);
    if (m.sa_flash) {   // tiled keys and values, split partials
      p.ks = take(cs * (size_t)m.H * m.tpadk * m.Es);
      p.vT = take(cs * (size_t)m.H * m.Es * m.tpadk);
      p.opart_s = take(4ul * m.sa_splits * Ht * m.Es);
      p.mpart_s = take(4ul * m.sa_splits * Ht * m.ns);
      p.lpart_s = take(4ul * m.sa_splits * Ht * m.ns);
    } else {
      p.ks = take(cs * Ht * m.Es);
      p.vT = take(cs * (size_t)m.H * m.Es * m.tpad);
      p.Ssa = take(4ul * (size_t)m.H * m.ns * m.t * m.tpad);
      p.Psa = take(cs * (size_t)m.H * m.ns * m.t * m.tpad);
    }
  }
  p.hid = take(cs * Ht * (m.F > 0 ? m.F : 1));
  p.total = (off > end1 ? off : end1) + 256;
  return p;
}

inline int grid1d(long n, int per = 256) {
  long b = (n + per - 1) / per;
  if (b > 65535L * 16) b = 65535L * 16;
  if (b < 1) b = 1;
  return (int)b;
}

// ---------------------------------------------------------------------------
// Validation of a layer's pointers
// ---------------------------------------------------------------------------
inline bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

inline still_status check_ptr(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(STILL_E_INVAL, "%s is NULL", name) : STILL_OK;
  if (misaligned(p)) return fail(STILL_E_INVAL, "%s is not 16-byte aligned", name);
  return STILL_OK;
}

inline still_status check_layer(const still_config* c, const Dims& m, const still_layer_weights* w, int layer) {
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

// One layer of the compaction (layer.hpp); IT = I/O type of K, V, weights and
// outputs, CT = MFMA operand / intermediate storage type.  Instantiated for
// (bf16, f16) and (float, float) in their own translation units.
template <class IT, class CT>
still_status run_layer(const still_config* cfg, const Dims& m, const Plan& p, char* ws, const still_layer_weights* w,
                       const void* Kp, const void* Vp, const double* positions, bool rerotate, void* Ckp, void* Cvp,
                       hipStream_t st);
extern template still_status run_layer<bf16, f16>(const still_config*, const Dims&, const Plan&, char*,
                                                  const still_layer_weights*, const void*, const void*,
                                                  const double*, bool, void*, void*, hipStream_t);
extern template still_status run_layer<float, float>(const still_config*, const Dims&, const Plan&, char*,
                                                     const still_layer_weights*, const void*, const void*,
                                                     const double*, bool, void*, void*, hipStream_t);

}  // namespace still
