/*
 * still.h - C ABI of the MI355X (gfx950) Still compactor forward pass.
 *
 * Still (arxiv 2606.07878) compacts one transformer layer's KV cache
 * (K, V in R^{H x N x d} per layer, keys RoPE-rotated by the base model) into
 * t << N synthetic entries (C_k, C_v in R^{H x t x d}) with a small per-layer
 * Perceiver (Section 2; Appendix A):
 *   1. RoPE-fix: keys are inverse-rotated into a position-free frame
 *      (Section 2.2; Appendix B, single-pass recipe step 3);
 *   2. X^(h) = [K^(h); V^(h)] in R^{N x 2d} (Appendix A, input concatenation);
 *   3. B pre-norm blocks on the latent bank Z in R^{H x t x d_l}:
 *        Z'   = Z   + CrossAttn(RMSNorm(Z), X)
 *        Z''  = Z'  + SelfAttn(RMSNorm(Z'))
 *        Z''' = Z'' + FFN(RMSNorm(Z''))            (Appendix A, blocks)
 *      cross-attention has n_c heads of width d_l each (expanded convention),
 *      biased Q/K projections, L2 QK-norm, the compactor's own RoPE (latent
 *      positions evenly spaced over [min p, max p]) and logits scaled by d_l;
 *   4. C_k = Z_out W_key, C_v = Z_out W_val (Appendix A, output projections);
 *   5. optional re-rotation of C_k at the latent (output) positions
 *      (Appendix B, single-pass recipe step 5).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor arguments are DEVICE pointers (memory allocated by the caller
 *   on the current HIP device), except the arrays of per-layer pointers of
 *   still_compact_model and the `blocks` array of still_layer_weights, which
 *   are HOST arrays holding device pointers.  The library never allocates or
 *   frees memory and keeps no device state between calls, except the static
 *   per-GPU array of still_attend_scratch (see there).
 * - Row-major, densely packed layouts.  Matrices are stored [out][in]
 *   (torch.nn.Linear layout): the paper's x W with W in R^{in x out} is
 *   evaluated as x W^T with the stored [out][in] array.
 * - Element type: STILL_MODE_BF16 -> every K, V, weight, bias, latent and
 *   output buffer holds bfloat16; STILL_MODE_FP32 -> float32 (validation
 *   mode: fp32 arithmetic, the near-maximal logits below in fp64).  Positions
 *   are always float64.
 * - Cross-attention logits (scaled by the head width, App. A) are computed
 *   from fp16 (bf16 mode) or fp32 operands; every key whose logit lies within
 *   10 log2 units of its latent's maximum is then recomputed accurately (fp32
 *   from split fp16 operands, or fp64) and its weight replaced.  Capacity: 256
 *   such keys per latent, from at most 1536 candidates per latent and key
 *   split.  Caches with more near-maximal keys per latent (rows repeated
 *   hundreds of times) exceed it and lose accuracy gradually.
 * - Work is enqueued on `stream` (NULL = default stream) and the call returns
 *   without synchronising.  Arguments are validated before anything is
 *   enqueued; a non-OK status means nothing was launched.  Faults during
 *   execution surface at the caller's next synchronisation.
 * - Outputs must not alias inputs or the workspace.  NaN/Inf in the inputs
 *   are not checked and propagate.
 * - Magnitudes, STILL_MODE_BF16: the MFMA operands are fp16 (max 65504).  The
 *   cache K, V may hold any finite bf16 value: each KV head is staged scaled
 *   by an exact power of two that brings its max |K|, |V| within 2^14 (1 for
 *   ordinary caches), undone on the value path.  Weights, biases and latents
 *   are converted to fp16 as they are and must lie within +-65504 (larger
 *   values overflow to +-inf and make the outputs non-finite).
 * - Calls that share a workspace must be ordered on one stream.
 */
#ifndef STILL_H_
#define STILL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  STILL_OK = 0,
  STILL_E_INVAL = -1,        /* NULL pointer, bad enum, non-positive size       */
  STILL_E_SHAPE = -2,        /* inconsistent shapes (e.g. t != latent bank size) */
  STILL_E_DTYPE = -3,        /* unknown mode                                     */
  STILL_E_WORKSPACE = -4,    /* workspace NULL or smaller than still_workspace_size */
  STILL_E_UNSUPPORTED = -5,  /* valid per the paper but not supported by these kernels */
  STILL_E_HIP = -6           /* a HIP runtime call failed (see still_last_error) */
} still_status;

/* Shapes the kernels take (anything else the paper allows returns
 * STILL_E_UNSUPPORTED): head_dim 64, 128 or 256; cross- and self-attention
 * head widths multiples of 128; latent_dim and ffn_hidden multiples of 8;
 * N * n_cross_heads * cross width * 2 and t * n_cross_heads * cross width * 2
 * below 2^32; H * N at most 128 * 65535; in bf16 mode at most 128 KV heads. */

typedef enum { STILL_MODE_BF16 = 0, STILL_MODE_FP32 = 1 } still_mode;
typedef enum { STILL_FFN_NONE = 0, STILL_FFN_SWIGLU = 1, STILL_FFN_GELU = 2 } still_ffn;

/* flags for the compaction calls */
enum { STILL_F_REROTATE = 1 };   /* re-rotate C_k at the output positions */

/* Hyper-parameters of one layer's compactor (Appendix A; canonical summary). */
typedef struct {
  int32_t n_kv_heads;        /* H, KV heads of the base model                         */
  int32_t head_dim;          /* d, base-model KV head width (even)                    */
  int32_t latent_dim;        /* D = d_l                                               */
  int32_t n_blocks;          /* B >= 1                                                */
  int32_t cross_every_block; /* 1: cross-attention in every block; 0: block 0 only    */
  int32_t n_cross_heads;     /* n_c >= 1                                              */
  int32_t cross_head_dim;    /* cross head width; 0 -> D (the paper's convention)     */
  int32_t n_self_heads;      /* n_s; 0 disables latent self-attention                 */
  int32_t self_head_dim;     /* self head width; 0 -> D                               */
  int32_t ffn_kind;          /* still_ffn                                             */
  int32_t ffn_hidden;        /* F, hidden width of the FFN                            */
  int32_t final_norm;        /* 1: RMSNorm before the output heads                    */
  float logit_scale_cross;   /* 0 -> cross head width (the d_l scale)                 */
  float logit_scale_self;    /* 0 -> self head width                                  */
  double compactor_rope_base;/* base of the compactor's internal RoPE (canonical 10)  */
  float rms_eps;             /* RMSNorm epsilon (1e-6)                                */
  float l2_eps;              /* QK-norm epsilon: x / max(||x||, l2_eps) (1e-12)       */
  int32_t mode;              /* still_mode                                            */
} still_config;

/* One block's parameters (device pointers; [out][in] matrices).  Tensors of
 * disabled sublayers are ignored and may be NULL.  A NULL bias means zero.
 *   E_c = n_c * cross_head_dim,  E_s = n_s * self_head_dim,  F = ffn_hidden
 *   ca_wq [E_c][D]  ca_bq [E_c]  ca_wk [E_c][2d]  ca_bk [E_c]
 *   ca_wv [E_c][2d] ca_wo [D][E_c]
 *   sa_wq [E_s][D]  sa_bq [E_s]  sa_wk [E_s][D]  sa_bk [E_s]
 *   sa_wv [E_s][D]  sa_wo [D][E_s]
 *   ffn_wg [F][D] ffn_wu [F][D] ffn_wd [D][F]   (GELU uses ffn_wu, ffn_wd) */
typedef struct {
  const void *ca_wq, *ca_bq, *ca_wk, *ca_bk, *ca_wv, *ca_wo;
  const void *sa_wq, *sa_bq, *sa_wk, *sa_bk, *sa_wv, *sa_wo;
  const void *ffn_wg, *ffn_wu, *ffn_wd;
} still_block_weights;

/* One layer's compactor: latent bank [H][t_bank][D], `blocks` is a HOST array
 * of n_blocks entries, output heads w_key, w_val [d][D]. */
typedef struct {
  const void *latents;
  int32_t t_bank;
  const still_block_weights *blocks;
  const void *w_key;
  const void *w_val;
} still_layer_weights;

/* Bytes of device workspace needed by a call compacting N tokens to t with
 * n_layers layers (the workspace is reused layer after layer).  Returns 0 if
 * the configuration is invalid or unsupported. */
size_t still_workspace_size(const still_config *cfg, int64_t N, int32_t t, int32_t n_layers);

/* Compact one layer.
 *   K, V        [H][N][d]  RoPE'd keys and values (device)
 *   positions   [N]        float64 logical cache positions (device); any real
 *                          values, not necessarily sorted or integral
 *   rope_theta             base of the base model's RoPE (un-rotation and
 *                          re-rotation use frequency theta^(-2j/d))
 *   t                      compact length; must equal w->t_bank
 *   flags                  STILL_F_REROTATE or 0
 *   C_k, C_v    [H][t][d]  outputs (device, caller-allocated)
 *   out_positions [t]      float64 output positions (device) or NULL:
 *                          p_min + i (p_max - p_min)/(t-1)  (p_min if t == 1)
 *   workspace              device buffer of >= still_workspace_size(cfg,N,t,1) bytes
 *   stream                 hipStream_t (NULL = default stream)           */
still_status still_compact_layer(const still_config *cfg, const still_layer_weights *w,
                                 const void *K, const void *V, const double *positions,
                                 int64_t N, double rope_theta, int32_t t, uint32_t flags,
                                 void *C_k, void *C_v, double *out_positions,
                                 void *workspace, size_t workspace_bytes, void *stream);

/* Compact n_layers independent layers (Appendix A, per-layer stack) that share
 * one position vector.  w, K, V, C_k, C_v are HOST arrays of n_layers entries
 * (each entry a device pointer, or a struct of device pointers for w). */
still_status still_compact_model(const still_config *cfg, int32_t n_layers,
                                 const still_layer_weights *w,
                                 const void *const *K, const void *const *V,
                                 const double *positions, int64_t N, double rope_theta,
                                 int32_t t, uint32_t flags,
                                 void *const *C_k, void *const *C_v, double *out_positions,
                                 void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Optional bias channel (Appendix A, output projections and beta shaping):
 * beta[h][i] = Z_out[h][i] . w_beta (Z_out = the final latent state, after the
 * final RMSNorm when cfg->final_norm), then optionally
 *   saturation      beta <- beta_max * tanh(beta / beta_max)     (beta_max > 0)
 *   mass matching   beta <- beta + mass_alpha * log(N / t) + log_x
 * in that order.  mass_alpha = 1, log_x = 0 is the uniform-attention offset;
 * log_x = log(x) is the learnable variant (x > 0); mass_alpha scales the
 * offset (the chunked-compaction sweep of the bias appendix).
 * ------------------------------------------------------------------------- */
typedef struct {
  float beta_max;      /* > 0: saturation; <= 0: off                      */
  float mass_alpha;    /* factor on log(N / t); 0: no uniform offset      */
  float log_x;         /* added as is; 0: none                            */
} still_beta_opts;

/* still_compact_model plus the bias channel.  w_beta: HOST array of n_layers
 * device pointers to [D] vectors (weight element type); beta: HOST array of
 * n_layers device [H][t] float32 outputs; beta_opts NULL = no shaping.  All
 * other arguments, errors and asynchrony as still_compact_model. */
still_status still_compact_model_beta(const still_config *cfg, int32_t n_layers,
                                      const still_layer_weights *w,
                                      const void *const *K, const void *const *V,
                                      const double *positions, int64_t N, double rope_theta,
                                      int32_t t, uint32_t flags,
                                      void *const *C_k, void *const *C_v, double *out_positions,
                                      const void *const *w_beta, const still_beta_opts *beta_opts,
                                      float *const *beta,
                                      void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Attention of base-model queries over a compacted prefix followed by an
 * uncompacted suffix, with the optional bias on the compact entries
 * (Appendix B, bias semantics in attention):
 *   out = sum_j exp(s_j) v_j / sum_j exp(s_j),
 *   s_j = scale q . C_k[j] + beta[j] for the t compact entries,
 *   s_j = scale q . K[j]              for the n_suffix suffix entries.
 * Keys are taken as stored (RoPE'd by the model when they were written).
 * Queries are taken as given, or, with rope_theta > 0, rotated here by the
 * base model's RoPE (rotate-half pairs (j, j + d/2), frequency
 * theta^(-2j/d), angles reduced in fp64) at q_positions: the logical
 * positions of the queries, i.e. their physical positions plus the offset
 * T - (physical prefix length) that a compacted cache carries (Appendix B,
 * logical vs physical cache length).  With causal = 1, query i of each query
 * head sits at suffix position n_suffix - n_queries + i and sees suffix keys
 * up to that position; all compact entries are visible to every query.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t n_kv_heads;   /* H                                                     */
  int32_t group;        /* query heads per KV head (grouped-query attention), >= 1 */
  int32_t head_dim;     /* d in {64, 128, 256}                                   */
  int32_t n_queries;    /* queries per query head; group * n_queries <= 32       */
  int32_t t;            /* compact entries per KV head, >= 0                     */
  int32_t n_suffix;     /* suffix entries per KV head, >= 0; t + n_suffix >= 1   */
  int32_t causal;       /* 0 or 1 (then n_suffix >= n_queries)                   */
  float scale;          /* logit scale; 0 -> 1/sqrt(d)                           */
  int32_t mode;         /* still_mode: element type of q, C_k, C_v, K, V, out    */
  double rope_theta;    /* > 0: rotate q at q_positions; 0: q used as given     */
} still_attend_config;

/* Bytes of device workspace still_attend needs (0: invalid configuration). */
size_t still_attend_workspace_size(const still_attend_config *cfg);

/*   q          [H*group][n_queries][d]  (query head h*group + g uses KV head h)
 *   q_positions [n_queries] fp64 logical positions (required iff rope_theta > 0)
 *   C_k, C_v   [H][t][d]         (NULL allowed when t = 0)
 *   beta       [H][t] float32    (NULL = no bias)
 *   K, V       [H][n_suffix][d]  (NULL allowed when n_suffix = 0)
 *   out        [H*group][n_queries][d]
 * All device pointers, 16-byte aligned; errors and asynchrony as the
 * compaction calls. */
still_status still_attend(const still_attend_config *cfg, const void *q, const double *q_positions,
                          const void *C_k, const void *C_v,
                          const float *beta, const void *K, const void *V, void *out,
                          void *workspace, size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * Backward pass of one layer's compactor (the training hot path without the
 * base model and its loss; Section 2.4 and Appendix E).  With upstream
 * gradients dC_k, dC_v of the layer's outputs, writes the gradient of
 *     L = <dC_k, C_k> + <dC_v, C_v>
 * with respect to every compactor tensor (the cache K, V gets none).
 *
 *   cfg            as for the forward pass; mode must be STILL_MODE_FP32
 *                  (all buffers float32), at most 8 blocks
 *   w, K, V, positions, N, rope_theta, t, flags   as still_compact_layer
 *   dC_k, dC_v     [H][t][d] float32 device buffers
 *   grad           a still_layer_weights of gradient OUTPUT buffers, one per
 *                  tensor of w with the same shape (float32, device):
 *                  grad->latents [H][t][D] (t_bank must equal t), the host
 *                  array grad->blocks[n_blocks], grad->w_key, grad->w_val.
 *                  A NULL entry skips that gradient.  Every non-NULL buffer
 *                  is overwritten (not accumulated into).
 *   C_k, C_v       optional [H][t][d] float32 outputs of the same forward
 *                  pass (NULL = not written)
 *   workspace      >= still_backward_workspace_size(cfg, N, t) bytes: the
 *                  forward intermediates kept for the chain rule, including
 *                  every attention probability (H n_c t N floats per
 *                  cross-attention block)
 * STILL_E_UNSUPPORTED in bf16 mode; other errors and asynchrony as the
 * compaction calls.
 * ------------------------------------------------------------------------- */
size_t still_backward_workspace_size(const still_config *cfg, int64_t N, int32_t t);
still_status still_compact_layer_backward(const still_config *cfg, const still_layer_weights *w, const void *K,
                                          const void *V, const double *positions, int64_t N, double rope_theta,
                                          int32_t t, uint32_t flags, const void *dC_k, const void *dC_v,
                                          const still_layer_weights *grad, void *C_k, void *C_v, void *workspace,
                                          size_t workspace_bytes, void *stream);

/* still_attend without a caller workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving (decode) loops,
 * harnesses that forbid allocation.  The split-N partials live in a
 * file-scope device array of STILL_ATTEND_SCRATCH_BYTES that every GPU the
 * library runs on holds until the process ends (its address is looked up once
 * per device, at the first call made with that device current).  The call
 * allocates nothing and frees nothing.
 *
 * Arguments, layouts, validation and asynchrony as still_attend.
 * STILL_E_WORKSPACE when still_attend_workspace_size(cfg) exceeds the array
 * (it never does for n_kv_heads <= 2048); STILL_E_HIP when the device or the
 * array's address cannot be obtained.  Every call on a GPU shares that GPU's
 * array: calls that overlap on one GPU (other streams, other threads) race
 * and must be ordered by the caller; the array keeps the last call's
 * contents, none of which a later call reads before writing it. */
enum { STILL_ATTEND_SCRATCH_BYTES = 68 << 20 };
still_status still_attend_scratch(const still_attend_config *cfg, const void *q, const double *q_positions,
                                  const void *C_k, const void *C_v, const float *beta, const void *K,
                                  const void *V, void *out, void *stream);

/* Human-readable name of a status code (static string). */
const char *still_status_string(int32_t status);

/* Detail of the last non-OK status returned on the calling thread. */
const char *still_last_error(void);

/* Optional event timing of the library's kernels, for benchmarks.
 * still_timing_enable(mask) makes every subsequent launch of a kernel class c
 * with bit (1 << c) set in mask record a hipEvent pair on its launch stream;
 * still_timing_enable(0) stops recording.  still_timing_read waits for the recorded events, returns
 * the summed duration (ms) and launch count of one class since the last
 * still_timing_reset, and may be called while the stream is idle only.
 * Event objects are created on first use and reused; nothing else is
 * allocated.  Not thread-safe: time one stream from one thread. */
enum {
  STILL_K_CROSS_ATTN = 0,   /* flash latent->cache cross-attention            */
  STILL_K_KPROJ = 1,        /* cross-attention key projection (+RoPE, norms)  */
  STILL_K_QPROJ = 2,        /* cross-attention query projection               */
  STILL_K_REFINE = 3,       /* exact-logit refinement of the top keys         */
  STILL_K_LATENT = 4,       /* latent-side GEMMs (V/O proj, self-attn, FFN, heads) */
  STILL_K_OTHER = 5,        /* norms, softmax, merge, tables, conversions, beta */
  STILL_K_ATTEND = 6,       /* still_attend: consumer attention and its merge  */
  STILL_K_STAGE = 7,        /* RoPE-fix staging of X, X^T: the KV-cache stream */
  STILL_K_COUNT = 8
};
still_status still_timing_enable(int32_t class_mask);
still_status still_timing_reset(void);
still_status still_timing_read(int32_t kernel_class, double *total_ms, int64_t *launches);

/* Library version string. */
const char *still_version(void);

#ifdef __cplusplus
}
#endif
#endif /* STILL_H_ */
