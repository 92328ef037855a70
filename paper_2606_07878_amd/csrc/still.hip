// still.hip - C ABI (include/still.h) of the Still compactor forward pass on
// MI355X: argument validation, the per-call tables, the layer loop and the
// consumer attention.  The per-layer launch sequences are compiled in
// layer_bf16.hip and layer_fp32.hip (layer.hpp).
#include "consumer.hpp"
#include "host.hpp"
#include "refine64.hpp"

#include <mutex>

namespace still {

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
  if (m.fp32) HIP_TRY(table(positions, m.N, m.dc, cbase, p.tab_ck));
  hipLaunchKernelGGL(inv_freq64_kernel, dim3((m.dc / 2 + 255) / 256), dim3(256), 0, st, cbase, m.dc,
                     (double*)(ws + p.invf_c));
  HIP_TRY(hipGetLastError());
  HIP_TRY(table(pq, m.t, m.dc, cbase, p.tab_cq));
  if (rerotate) HIP_TRY(table(pq, m.t, m.d, rope_theta, p.tab_bq));
  hipLaunchKernelGGL(inv_freq64_kernel, dim3((m.d / 2 + 255) / 256), dim3(256), 0, st, rope_theta, m.d,
                     (double*)(ws + p.invf_b));
  HIP_TRY(hipGetLastError());
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
    s = m.fp32 ? run_layer<float, float>(cfg, m, p, ws, &w[l], K[l], V[l], positions, rerot, Ck[l], Cv[l], st)
               : run_layer<bf16, f16>(cfg, m, p, ws, &w[l], K[l], V[l], positions, rerot, Ck[l], Cv[l], st);
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

// ---------------------------------------------------------------------------
// Scratch of still_attend_scratch: the split partials of one call, in a
// file-scope device array (one copy per GPU).  Host code uses the address
// hipGetSymbolAddress returns for the current device, never the array's name.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[STILL_ATTEND_SCRATCH_BYTES];
constexpr int SCRATCH_MAX_DEVICES = 64;
static void* scratch_ptr[SCRATCH_MAX_DEVICES];
static std::mutex scratch_mu;

static still_status scratch_for_current_device(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return fail(STILL_E_UNSUPPORTED, "device %d beyond %d", dev,
                                                         SCRATCH_MAX_DEVICES);
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(STILL_E_HIP, "hipGetSymbolAddress returned NULL for the scratch array");
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return STILL_OK;
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

still_status still_attend_scratch(const still_attend_config* cfg, const void* q, const double* q_positions,
                                  const void* C_k, const void* C_v, const float* beta, const void* K, const void* V,
                                  void* out, void* stream) {
  AttendPlan ap;
  still_status s = attend_plan(cfg, &ap);
  if (s != STILL_OK) return s;
  if (ap.total > (size_t)STILL_ATTEND_SCRATCH_BYTES)
    return fail(STILL_E_WORKSPACE, "attend needs %zu bytes of scratch; the static array holds %zu", ap.total,
                (size_t)STILL_ATTEND_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((s = scratch_for_current_device(&ws)) != STILL_OK) return s;
  return still_attend(cfg, q, q_positions, C_k, C_v, beta, K, V, out, ws, (size_t)STILL_ATTEND_SCRATCH_BYTES, stream);
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
