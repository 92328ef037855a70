// consumer.hpp - attention of base-model queries over a compacted cache
// followed by an uncompacted suffix, with the optional per-entry bias of the
// compact part (Appendix B, bias semantics in attention):
//   out = sum_j exp(s_j) v_j / sum_j exp(s_j),
//   s_j = scale q.C_k[j] + beta[j]  (j < t),   s_j = scale q.K[j - t]  (suffix).
// Decode-shaped (a few query rows per KV head): one wave per (KV head, key
// split), lane = key for the logits, lane = feature for P.V, online softmax
// over 64-key chunks; splits merged by a second kernel.  fp32 arithmetic.
#pragma once
#include "common.hpp"
#include "misc.hpp"

namespace still {

constexpr int ATTEND_MAX_ROWS = 32;   // group * n_queries
constexpr int ATTEND_CHUNKS = 4;      // 64-key chunks per split

struct ConsumerArgs {
  const void* q;        // [H*group][nq][D]
  const void* ck;       // [H][t][D]
  const void* cv;
  const float* beta;    // [H][t] or NULL
  const void* k;        // [H][S][D] suffix keys (RoPE'd), may be NULL when S = 0
  const void* v;
  void* out;            // [H*group][nq][D]
  float* opart;         // [splits][H][R][D]
  float* mpart;         // [splits][H][R]
  float* lpart;
  int H, group, nq, t, S, causal, splits;
  float scale;
};

template <class T> __device__ __forceinline__ float ld1(const T* p) { return to_f32(*p); }

template <class IT, int D>
__global__ __launch_bounds__(64) void attend_partial_kernel(ConsumerArgs a) {
  constexpr int FPL = D / 64;                 // features per lane in P.V
  __shared__ float qs[ATTEND_MAX_ROWS][D];    // query rows, fp32
  __shared__ float ps[64][ATTEND_MAX_ROWS];   // chunk probabilities [key][row]
  const int lane = threadIdx.x;
  const int split = blockIdx.x, h = blockIdx.y;
  const int R = a.group * a.nq, total = a.t + a.S;
  const int j0 = split * (64 * ATTEND_CHUNKS);
  const IT* qh = (const IT*)a.q + (long)h * a.group * a.nq * D;   // rows g*nq + i are contiguous
  for (int e = lane; e < R * D; e += 64) qs[e / D][e % D] = ld1(qh + e);
  __syncthreads();

  float m[ATTEND_MAX_ROWS], l[ATTEND_MAX_ROWS], o[ATTEND_MAX_ROWS][FPL];
#pragma unroll
  for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int u = 0; u < FPL; ++u) o[r][u] = 0.f;
  }
  for (int c = 0; c < ATTEND_CHUNKS; ++c) {
    const int jb = j0 + 64 * c;
    if (jb >= total) break;
    // ---- logits: lane = key
    const int j = jb + lane;
    float s[ATTEND_MAX_ROWS];
#pragma unroll
    for (int r = 0; r < ATTEND_MAX_ROWS; ++r) s[r] = 0.f;
    if (j < total) {
      const IT* kr = j < a.t ? (const IT*)a.ck + ((long)h * a.t + j) * D
                             : (const IT*)a.k + ((long)h * a.S + (j - a.t)) * D;
      for (int f = 0; f < D; f += 8) {
        float kv[8];
        load8(kr + f, kv);   // 16-byte run of the key row
#pragma unroll
        for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
          if (r < R) {
            const float4 q0 = *(const float4*)&qs[r][f], q1 = *(const float4*)&qs[r][f + 4];
            s[r] += q0.x * kv[0] + q0.y * kv[1] + q0.z * kv[2] + q0.w * kv[3] + q1.x * kv[4] + q1.y * kv[5] +
                    q1.z * kv[6] + q1.w * kv[7];
          }
        }
      }
    }
    const float bj = (j < a.t && a.beta) ? a.beta[(long)h * a.t + j] : 0.f;
#pragma unroll
    for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
      if (r >= R) continue;
      bool ok = j < total;
      if (ok && a.causal && j >= a.t) {   // row r = g*nq + i sits at suffix position S - nq + i
        const int i = r % a.nq;
        ok = (j - a.t) <= a.S - a.nq + i;
      }
      s[r] = ok ? s[r] * a.scale + bj : -INFINITY;
    }
    // ---- online softmax per row over the chunk
#pragma unroll
    for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
      if (r >= R) continue;
      float cm = s[r];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off));
      const float mn = fmaxf(m[r], cm);
      const float mref = mn == -INFINITY ? 0.f : mn;
      const float p = expf(s[r] - mref);
      float cs = p;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) cs += __shfl_xor(cs, off);
      const float al = expf(m[r] - mref);
      l[r] = l[r] * al + cs;
#pragma unroll
      for (int u = 0; u < FPL; ++u) o[r][u] *= al;
      m[r] = mn;
      ps[lane][r] = p;
    }
    __syncthreads();
    // ---- P.V: lane = features [lane*FPL, (lane+1)*FPL)
    const int nk = min(64, total - jb);
    for (int kk = 0; kk < nk; ++kk) {
      const int jj = jb + kk;
      const IT* vr = jj < a.t ? (const IT*)a.cv + ((long)h * a.t + jj) * D
                              : (const IT*)a.v + ((long)h * a.S + (jj - a.t)) * D;
      float vv[FPL];
#pragma unroll
      for (int u = 0; u < FPL; ++u) vv[u] = ld1(vr + lane * FPL + u);
#pragma unroll
      for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
        if (r >= R) continue;
        const float p = ps[kk][r];
#pragma unroll
        for (int u = 0; u < FPL; ++u) o[r][u] += p * vv[u];
      }
    }
    __syncthreads();
  }
  // ---- split partials
  const long base = (long)split * a.H + h;
#pragma unroll
  for (int r = 0; r < ATTEND_MAX_ROWS; ++r) {
    if (r >= R) continue;
    float* op = a.opart + (base * ATTEND_MAX_ROWS + r) * D + lane * FPL;
#pragma unroll
    for (int u = 0; u < FPL; ++u) op[u] = o[r][u];
    if (lane == 0) {
      a.mpart[base * ATTEND_MAX_ROWS + r] = m[r];
      a.lpart[base * ATTEND_MAX_ROWS + r] = l[r];
    }
  }
}

// out[row] = sum_s exp(m_s - M) O_s / sum_s exp(m_s - M) l_s, one wave per (KV head, row)
template <class IT, int D>
__global__ __launch_bounds__(64) void attend_merge_kernel(ConsumerArgs a) {
  constexpr int FPL = D / 64;
  const int lane = threadIdx.x;
  const int r = blockIdx.x, h = blockIdx.y;
  float M = -INFINITY;
  for (int s = 0; s < a.splits; ++s) M = fmaxf(M, a.mpart[((long)s * a.H + h) * ATTEND_MAX_ROWS + r]);
  const float mref = M == -INFINITY ? 0.f : M;
  float L = 0.f, acc[FPL];
#pragma unroll
  for (int u = 0; u < FPL; ++u) acc[u] = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const long b = ((long)s * a.H + h) * ATTEND_MAX_ROWS + r;
    const float w = expf(a.mpart[b] - mref);
    L += w * a.lpart[b];
#pragma unroll
    for (int u = 0; u < FPL; ++u) acc[u] += w * a.opart[b * D + lane * FPL + u];
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  IT* dst = (IT*)a.out + ((long)h * a.group * a.nq + r) * D + lane * FPL;
#pragma unroll
  for (int u = 0; u < FPL; ++u) dst[u] = from_f32<IT>(acc[u] * inv);
}

// beta[h][i] = shape(Z_out[h*t + i] . w_beta), Z_out = Z or RMSNorm(Z); one wave per row.
struct BetaShape {
  float beta_max;     // > 0: beta_max * tanh(beta / beta_max)
  float offset;       // added last (mass matching: log(N / t) + log_x; else 0)
};

template <class WT>
__global__ __launch_bounds__(256) void beta_kernel(const float* __restrict__ Z, const WT* __restrict__ w,
                                                   long rows, int D, int final_norm, float eps, BetaShape sh,
                                                   float* __restrict__ beta) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* z = Z + row * D;
  float dot = 0.f, ss = 0.f;
  for (int i = lane; i < D; i += 64) {
    dot += z[i] * to_f32(w[i]);
    ss += z[i] * z[i];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    dot += __shfl_xor(dot, o);
    ss += __shfl_xor(ss, o);
  }
  if (lane == 0) {
    float b = final_norm ? dot / sqrtf(ss / (float)D + eps) : dot;
    if (sh.beta_max > 0.f) b = sh.beta_max * tanhf(b / sh.beta_max);
    beta[row] = b + sh.offset;
  }
}

}  // namespace still
