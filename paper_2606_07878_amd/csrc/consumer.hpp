// consumer.hpp - attention of base-model queries over a compacted cache
// followed by an uncompacted suffix, with the optional per-entry bias of the
// compact part (Appendix B, bias semantics in attention):
//   out = sum_j exp(s_j) v_j / sum_j exp(s_j),
//   s_j = scale q.C_k[j] + beta[j]  (j < t),   s_j = scale q.K[j - t]  (suffix).
// Decode-shaped (a few query rows per KV head): one wave per (KV head, key
// split), 64-key chunks with 16-byte loads; lane = key for the logits,
// lane = feature for P.V with the V rows staged in LDS; online softmax over
// the chunks; splits merged by a second kernel.  fp32 arithmetic.
#pragma once
#include "common.hpp"
#include "misc.hpp"

namespace still {

constexpr int ATTEND_MAX_ROWS = 32;   // group * n_queries
constexpr int ATTEND_DECODE_ROWS = 8; // at most this many rows: the register-resident decode kernel
constexpr int ATTEND_KC = 64;         // keys per chunk: one per lane for the logits

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
  int H, group, nq, t, S, causal, splits, cps;   // cps: chunks per split
  float scale;
  const double* qpos;   // [nq] logical query positions, or NULL (q as given)
  double theta;         // base RoPE theta when qpos is set
};

// Rotation angle of feature pair jh (< d/2) at position pos, reduced to
// [-pi, pi] in fp64 before the fp32 sine and cosine (positions reach 1e5+).
__device__ __forceinline__ void rope_angle(double pos, int jh, int d, double theta, float& c, float& s) {
  const double inv = pow(theta, -2.0 * jh / d);
  double phi = pos * inv;
  phi -= 6.283185307179586 * rint(phi * 0.15915494309189535);
  sincosf((float)phi, &s, &c);
}

// Per-(element type, head width) tiling of one chunk.  A key row is PPR
// 16-byte pieces; the V rows of a chunk are staged through LDS VROWS at a
// time so that a lane holds at most 16 pieces in flight; K rows are read
// lane = key, KSLAB pieces per round trip.
template <class IT, int D>
struct AttendTile {
  static constexpr int ROWB = D * (int)sizeof(IT);
  static constexpr int PPR = ROWB / 16;
  static constexpr int EPP = 16 / (int)sizeof(IT);        // elements per piece
  static constexpr int VROWS = 16384 / ROWB < ATTEND_KC ? 16384 / ROWB : ATTEND_KC;
  static constexpr int VPL = VROWS * PPR / 64;             // V pieces per lane per pass
  static constexpr int KSLAB = PPR < 16 ? PPR : 16;
  static constexpr int FPL = D / 64;                       // output features per lane
  static_assert(VROWS * PPR % 64 == 0 && PPR % KSLAB == 0, "tile shape");
};

// dynamic LDS: q rows fp32 [RB][D] (rows past R zero) | V pass [VROWS][ROWB] | P [64][RB]
template <class IT, int D>
inline size_t attend_lds_bytes(int RB) {
  using TL = AttendTile<IT, D>;
  return (size_t)RB * D * 4 + (size_t)TL::VROWS * TL::ROWB + (size_t)ATTEND_KC * RB * 4;
}

// 16-byte pieces as a native vector: plain loads and stores (a HIP uint4 copy
// lowers to memcpy, which keeps a staged array in scratch memory)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <class T> __device__ __forceinline__ void unpack16(const u32x4& u, float (&o)[16 / sizeof(T)]);
template <> __device__ __forceinline__ void unpack16<bf16>(const u32x4& u, float (&o)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <> __device__ __forceinline__ void unpack16<float>(const u32x4& u, float (&o)[4]) {
  o[0] = __uint_as_float(u.x);
  o[1] = __uint_as_float(u.y);
  o[2] = __uint_as_float(u.z);
  o[3] = __uint_as_float(u.w);
}

// Chunk c of KV head h: chunks [0, nck) cover the compact rows, [nck, nck + nsk)
// the suffix rows; a chunk never straddles the two, so its base pointer and row
// count are wave-uniform.
struct AttendChunk {
  const char* kbase;   // row 0 of this part's keys for head h
  const char* vbase;
  int j0, rows;        // first row of the chunk within the part, rows in the part
  bool compact;
};

template <class IT, int D>
__device__ __forceinline__ AttendChunk attend_chunk(const ConsumerArgs& a, int h, int c) {
  constexpr long ROWB = (long)D * sizeof(IT);
  const int nck = (a.t + ATTEND_KC - 1) / ATTEND_KC;
  AttendChunk k;
  k.compact = c < nck;
  k.rows = k.compact ? a.t : a.S;
  k.j0 = (k.compact ? c : c - nck) * ATTEND_KC;
  const long hoff = (long)h * k.rows * ROWB;
  k.kbase = (const char*)(k.compact ? a.ck : a.k) + hoff;
  k.vbase = (const char*)(k.compact ? a.cv : a.v) + hoff;
  return k;
}

template <class IT, int D>
__device__ __forceinline__ void attend_load_v(const AttendChunk& ch, int vb, int lane,
                                              u32x4 (&vp)[AttendTile<IT, D>::VPL]) {
  using TL = AttendTile<IT, D>;
#pragma unroll
  for (int i = 0; i < TL::VPL; ++i) {
    const int pc = lane + 64 * i, row = pc / TL::PPR, col = pc % TL::PPR;
    vp[i] = ((const u32x4*)(ch.vbase + (long)min(ch.j0 + vb + row, ch.rows - 1) * TL::ROWB))[col];
  }
}

// Query rows R > 8 (prefill-shaped calls): lane = key for the logits with the
// query rows read from LDS, lane = features for P.V with V staged in LDS and
// the probabilities exchanged through LDS.  RB: bound on R (register arrays).
template <class IT, int D, int RB>
__global__ __launch_bounds__(64) void attend_partial_kernel(ConsumerArgs a) {
  using TL = AttendTile<IT, D>;
  constexpr int FPL = TL::FPL;
  extern __shared__ float4 attend_smem[];
  const int R = a.group * a.nq;
  float* qs = (float*)attend_smem;                                   // [RB][D]
  char* vs = (char*)(qs + RB * D);                                    // [VROWS][ROWB]
  float* ps = (float*)(vs + TL::VROWS * TL::ROWB);                    // [64][RB]
  const int lane = threadIdx.x;
  const int split = blockIdx.x, h = blockIdx.y;
  const int nchunks = (a.t + ATTEND_KC - 1) / ATTEND_KC + (a.S + ATTEND_KC - 1) / ATTEND_KC;
  const int c0 = split * a.cps, c1 = min(nchunks, c0 + a.cps);   // this split's chunks [c0, c1)
  {  // query rows g*nq + i of KV head h are contiguous: 16-byte pieces, fp32 in LDS
    const u32x4* qh = (const u32x4*)((const IT*)a.q + (long)h * R * D);
    const int np = R * D / TL::EPP;
#pragma unroll 4
    for (int pc = lane; pc < np; pc += 64) {
      float f[TL::EPP];
      unpack16<IT>(qh[pc], f);
#pragma unroll
      for (int e = 0; e < TL::EPP; e += 4)
        *(float4*)&qs[pc * TL::EPP + e] = make_float4(f[e], f[e + 1], f[e + 2], f[e + 3]);
    }
  }
  __syncthreads();
  if (a.qpos) {  // RoPE of the query rows at their logical positions (rotate-half pairs)
    constexpr int HD = D / 2;
    for (int e = lane; e < R * HD; e += 64) {
      const int r = e / HD, j = e % HD;
      float c, sn;
      rope_angle(a.qpos[r % a.nq], j, D, a.theta, c, sn);
      const float x0 = qs[r * D + j], x1 = qs[r * D + j + HD];
      qs[r * D + j] = x0 * c - x1 * sn;
      qs[r * D + j + HD] = x1 * c + x0 * sn;
    }
    __syncthreads();
  }

  float m[RB], l[RB], o[RB][FPL];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int u = 0; u < FPL; ++u) o[r][u] = 0.f;
  }
  for (int c = c0; c < c1; ++c) {
    const AttendChunk ch = attend_chunk<IT, D>(a, h, c);
    // ---- logits, lane = key (row jl of the part; rows past its end are clamped and masked)
    const int jl = ch.j0 + lane;
    const u32x4* kr = (const u32x4*)(ch.kbase + (long)min(jl, ch.rows - 1) * TL::ROWB);
    float s[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) s[r] = 0.f;
#pragma unroll
    for (int sb = 0; sb < TL::PPR; sb += TL::KSLAB) {
      u32x4 kp[TL::KSLAB];
#pragma unroll
      for (int i = 0; i < TL::KSLAB; ++i) kp[i] = kr[sb + i];
#pragma unroll
      for (int i = 0; i < TL::KSLAB; ++i) {
        float kv[TL::EPP];
        unpack16<IT>(kp[i], kv);
        const int f0 = (sb + i) * TL::EPP;
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          if (r < R) {
#pragma unroll
            for (int e = 0; e < TL::EPP; e += 4) {
              const float4 qv = *(const float4*)&qs[r * D + f0 + e];
              s[r] += qv.x * kv[e] + qv.y * kv[e + 1] + qv.z * kv[e + 2] + qv.w * kv[e + 3];
            }
          }
        }
      }
    }
    const bool valid = jl < ch.rows;
    const float bj = (ch.compact && valid && a.beta) ? a.beta[(long)h * a.t + jl] : 0.f;
    // ---- online softmax per row over the chunk; P to LDS
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      if (r >= R) continue;
      const bool ok = valid && (ch.compact || !a.causal || jl <= a.S - a.nq + r % a.nq);   // row g*nq+i
      const float sv = ok ? s[r] * a.scale + bj : -INFINITY;
      float cm = sv;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off));
      const float mn = fmaxf(m[r], cm);
      const float mref = mn == -INFINITY ? 0.f : mn;
      const float p = expf(sv - mref);
      float cs = p;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) cs += __shfl_xor(cs, off);
      const float al = expf(m[r] - mref);
      l[r] = l[r] * al + cs;
#pragma unroll
      for (int u = 0; u < FPL; ++u) o[r][u] *= al;
      m[r] = mn;
      ps[lane * RB + r] = p;
    }
    // ---- P.V through LDS, VROWS rows per pass; lane = features [lane*FPL, (lane+1)*FPL)
#pragma unroll
    for (int vb = 0; vb < ATTEND_KC; vb += TL::VROWS) {
      u32x4 vp[TL::VPL];
      attend_load_v<IT, D>(ch, vb, lane, vp);
      __syncthreads();   // previous readers of vs are done; ps is complete
#pragma unroll
      for (int i = 0; i < TL::VPL; ++i) ((u32x4*)vs)[lane + 64 * i] = vp[i];
      __syncthreads();
#pragma unroll 4
      for (int kk = 0; kk < TL::VROWS; ++kk) {
        float vv[FPL];
        const IT* vrow = (const IT*)(vs + kk * TL::ROWB) + lane * FPL;
#pragma unroll
        for (int u = 0; u < FPL; ++u) vv[u] = to_f32(vrow[u]);
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          if (r >= R) continue;
          const float p = ps[(vb + kk) * RB + r];
#pragma unroll
          for (int u = 0; u < FPL; ++u) o[r][u] += p * vv[u];
        }
      }
    }
    __syncthreads();   // ps and vs are rewritten by the next chunk
  }
  // ---- split partials
  const long base = ((long)split * a.H + h) * R;
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    if (r >= R) continue;
    float* op = a.opart + (base + r) * D + lane * FPL;
#pragma unroll
    for (int u = 0; u < FPL; ++u) op[u] = o[r][u];
    if (lane == 0) {
      a.mpart[base + r] = m[r];
      a.lpart[base + r] = l[r];
    }
  }
}

// ---------------------------------------------------------------------------
// Decode-shaped attention (R <= 8 query rows per KV head), no LDS in the chunk
// loop.  A key row is PPR 16-byte pieces; LPK = PPR lanes share one key (lane
// piece pl = lane % LPK holds features [pl*EPP, (pl+1)*EPP)), KPI = 64 / LPK
// keys are read per instruction, NIT instructions make a chunk of KC keys.
// Each lane keeps its slice of every query row in registers; a dot product is
// the lane's EPP-term partial summed over its LPK lanes by DPP row operations
// and, past 16 lanes, shuffles.  The lane then holds the probability of its own
// key, so P.V accumulates o[r][its features] without any exchange; the KPI key
// slots are summed once per split.
// ---------------------------------------------------------------------------
template <class IT, int D, int RB>
struct DecodeTile {
  static constexpr int PPR = D * (int)sizeof(IT) / 16;
  static constexpr int LPK = PPR;
  static constexpr int KPI = 64 / LPK;
  static constexpr int EPP = 16 / (int)sizeof(IT);
  static constexpr int NIT = RB <= 4 ? 8 : 4;
  static constexpr int KC = NIT * KPI;
  static_assert(LPK >= 8 && LPK <= 64, "lanes per key");
};

// sum over aligned groups of N lanes (N in 8, 16, 32, 64); every lane gets its group's sum
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));   // xor 1
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));   // xor 2
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));  // half-row mirror
  if constexpr (N >= 16)
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));  // row mirror
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

// combine over the key slots: lanes l, l ^ LPK, l ^ 2 LPK, ... (same piece position)
template <int LPK>
__device__ __forceinline__ float slots_max(float x) {
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
template <int LPK>
__device__ __forceinline__ float slots_sum(float x) {
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) x += __shfl_xor(x, off);
  return x;
}

template <class IT, int D, int RB>
struct DecodeStage {
  u32x4 k[DecodeTile<IT, D, RB>::NIT];
  u32x4 v[DecodeTile<IT, D, RB>::NIT];
  float b[DecodeTile<IT, D, RB>::NIT];
};

template <class IT, int D, int RB>
__device__ __forceinline__ void decode_load(const ConsumerArgs& a, const AttendChunk& ch, int h, int lane,
                                            DecodeStage<IT, D, RB>& st) {
  using TL = DecodeTile<IT, D, RB>;
  constexpr long ROWB = (long)D * sizeof(IT);
  const int g = lane / TL::LPK, pl = lane % TL::LPK;
#pragma unroll
  for (int it = 0; it < TL::NIT; ++it) {
    const int jl = min(ch.j0 + it * TL::KPI + g, ch.rows - 1);
    st.k[it] = ((const u32x4*)(ch.kbase + jl * ROWB))[pl];
    st.v[it] = ((const u32x4*)(ch.vbase + jl * ROWB))[pl];
    st.b[it] = (ch.compact && a.beta) ? a.beta[(long)h * a.t + jl] : 0.f;
  }
}

template <class IT, int D, int RB>
__global__ __launch_bounds__(64) void attend_decode_kernel(ConsumerArgs a) {
  using TL = DecodeTile<IT, D, RB>;
  constexpr int EPP = TL::EPP, NIT = TL::NIT;
  const int lane = threadIdx.x, g = lane / TL::LPK, pl = lane % TL::LPK;
  const int split = blockIdx.x, h = blockIdx.y, R = a.group * a.nq;
  const int nck = (a.t + TL::KC - 1) / TL::KC;
  const int nchunks = nck + (a.S + TL::KC - 1) / TL::KC;
  const int c0 = split * a.cps, c1 = min(nchunks, c0 + a.cps);
  auto chunk = [&](int c) {
    AttendChunk k;
    k.compact = c < nck;
    k.rows = k.compact ? a.t : a.S;
    k.j0 = (k.compact ? c : c - nck) * TL::KC;
    const long hoff = (long)h * k.rows * D * (long)sizeof(IT);
    k.kbase = (const char*)(k.compact ? a.ck : a.k) + hoff;
    k.vbase = (const char*)(k.compact ? a.cv : a.v) + hoff;
    return k;
  };

  DecodeStage<IT, D, RB> cur, nxt;
  decode_load<IT, D, RB>(a, chunk(c0), h, lane, cur);
  // the lane's slice of every query row (rows past R repeat row R-1 and are never stored)
  float qv[RB][EPP];
  int lim[RB];
  {
    const IT* qh = (const IT*)a.q + (long)h * R * D;
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int rr = min(r, R - 1);
      unpack16<IT>(((const u32x4*)(qh + (long)rr * D))[pl], qv[r]);
      lim[r] = a.causal ? a.S - a.nq + rr % a.nq : 0x7fffffff;   // row g*nq+i sees suffix rows <= S-nq+i
    }
    if (a.qpos) {  // RoPE at the logical positions: the pair partner of feature j sits LPK/2 lanes away
      const bool upper = pl >= TL::LPK / 2;
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const double pos = a.qpos[min(r, R - 1) % a.nq];
#pragma unroll
        for (int e = 0; e < EPP; ++e) {
          const float other = __shfl_xor(qv[r][e], TL::LPK / 2);
          float c, sn;
          rope_angle(pos, (pl % (TL::LPK / 2)) * EPP + e, D, a.theta, c, sn);
          qv[r][e] = upper ? qv[r][e] * c + other * sn : qv[r][e] * c - other * sn;
        }
      }
    }
  }
  float m[RB], l[RB], o[RB][EPP];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < EPP; ++e) o[r][e] = 0.f;
  }
  for (int c = c0; c < c1; ++c) {
    const AttendChunk ch = chunk(c);
    decode_load<IT, D, RB>(a, chunk(min(c + 1, c1 - 1)), h, lane, nxt);   // one chunk ahead, in bounds
    float lg[NIT][RB];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      float kv[EPP];
      unpack16<IT>(cur.k[it], kv);
      const int jl = ch.j0 + it * TL::KPI + g;
      const bool valid = jl < ch.rows;
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPP; ++e) d += qv[r][e] * kv[e];
        d = group_sum<TL::LPK>(d);
        const bool ok = valid && (ch.compact || jl <= lim[r]);
        lg[it][r] = ok ? d * a.scale + cur.b[it] : -INFINITY;
      }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      float cm = lg[0][r];
#pragma unroll
      for (int it = 1; it < NIT; ++it) cm = fmaxf(cm, lg[it][r]);
      cm = slots_max<TL::LPK>(cm);
      const float mn = fmaxf(m[r], cm);
      const float mref = mn == -INFINITY ? 0.f : mn;
      float cs = 0.f;
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        lg[it][r] = expf(lg[it][r] - mref);
        cs += lg[it][r];
      }
      cs = slots_sum<TL::LPK>(cs);   // lanes of one slot hold the same keys: sum over the slots
      const float al = expf(m[r] - mref);
      l[r] = l[r] * al + cs;
      m[r] = mn;
#pragma unroll
      for (int e = 0; e < EPP; ++e) o[r][e] *= al;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      float vv[EPP];
      unpack16<IT>(cur.v[it], vv);
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int e = 0; e < EPP; ++e) o[r][e] += lg[it][r] * vv[e];
    }
    cur = nxt;
  }
  // sum the key slots; lanes of slot 0 write the split's partial rows
  const long base = ((long)split * a.H + h) * R;
#pragma unroll
  for (int r = 0; r < RB; ++r) {
#pragma unroll
    for (int e = 0; e < EPP; ++e) o[r][e] = slots_sum<TL::LPK>(o[r][e]);
    if (r < R && g == 0) {
      float* op = a.opart + (base + r) * D + pl * EPP;
#pragma unroll
      for (int e = 0; e < EPP; e += 4) *(float4*)(op + e) = make_float4(o[r][e], o[r][e + 1], o[r][e + 2], o[r][e + 3]);
      if (pl == 0) {
        a.mpart[base + r] = m[r];
        a.lpart[base + r] = l[r];
      }
    }
  }
}

// out[row] = sum_s exp(m_s - M) O_s / sum_s exp(m_s - M) l_s.  One block of
// ATTEND_MERGE_WAVES waves per (row, KV head): wave w takes splits w, w + W,
// ...; every lane holds FPL features; the waves' maxima, sums and rows are
// combined through LDS.
constexpr int ATTEND_MERGE_WAVES = 8;

template <class IT, int D>
__global__ __launch_bounds__(64 * ATTEND_MERGE_WAVES) void attend_merge_kernel(ConsumerArgs a) {
  constexpr int FPL = D / 64, W = ATTEND_MERGE_WAVES;
  __shared__ float red[W];
  __shared__ float racc[W][D];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int r = blockIdx.x, h = blockIdx.y, R = a.group * a.nq;
  const long stride = (long)a.H * R;   // between consecutive splits
  const long b0 = (long)h * R + r;
  float M = -INFINITY;
  for (int s = threadIdx.x; s < a.splits; s += 64 * W) M = fmaxf(M, a.mpart[s * stride + b0]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  if (lane == 0) red[wv] = M;
  __syncthreads();
  M = red[0];
#pragma unroll
  for (int i = 1; i < W; ++i) M = fmaxf(M, red[i]);
  const float mref = M == -INFINITY ? 0.f : M;
  float L = 0.f, acc[FPL];
#pragma unroll
  for (int u = 0; u < FPL; ++u) acc[u] = 0.f;
#pragma unroll 4
  for (int s = wv; s < a.splits; s += W) {
    const long b = s * stride + b0;
    const float w = expf(a.mpart[b] - mref);
    L += w * a.lpart[b];
    const float* op = a.opart + b * D + lane * FPL;
#pragma unroll
    for (int u = 0; u < FPL; ++u) acc[u] += w * op[u];
  }
#pragma unroll
  for (int u = 0; u < FPL; ++u) racc[wv][lane * FPL + u] = acc[u];
  __syncthreads();
  if (lane == 0) red[wv] = L;   // every lane of a wave holds the same L
  __syncthreads();
  if (wv == 0) {
    float Lt = 0.f;
#pragma unroll
    for (int i = 0; i < W; ++i) Lt += red[i];
    const float inv = Lt > 0.f ? 1.f / Lt : 0.f;
    IT* dst = (IT*)a.out + b0 * D + lane * FPL;
#pragma unroll
    for (int u = 0; u < FPL; ++u) {
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < W; ++i) v += racc[i][lane * FPL + u];
      dst[u] = from_f32<IT>(v * inv);
    }
  }
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
