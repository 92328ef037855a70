// refine.hpp - exact logits of the refined keys on the fp16 path, one kernel:
// gather of the keys' RoPE-fixed rows, their key projection and the dot
// product with the query.
//
// For the candidate slot (latent i, key n) of a (KV head h, cross head c)
// pair the refinement needs the key's projected row k~ = W_K x_n + b_K (its
// sum of squares for the QK-norm) and the dot product of the compactor-RoPE
// rotated k~ with the query row q~_i.  The key row is carried at better than
// fp16 precision as x_n = [K_hi | V | K_lo] (the RoPE-fixed key split into
// two fp16 parts), contracted with [W_K | W_K(key half)]: one 3d-wide MFMA
// product per slot, in which each W_K fragment of the key half serves both
// the K_hi and the K_lo columns (2d columns of W_K streamed per row tile).
//
// Workgroup = BM candidate rows of one (h, c) list x all dc output widths.
// The rows are gathered (base-RoPE un-rotation, hi/lo split) straight into
// LDS, where they stay for the whole workgroup.  The product is computed
// transposed, k~^T = W_K x^T (MFMA rows = output widths, columns =
// candidates): lane l of an accumulator then holds candidate l % 32 and 16
// widths in runs of 4, so the query values it needs are
// 16-byte vector loads (the compactor-RoPE rotation of each candidate's key
// position is computed in place from the fp64 position and frequencies) and
// the per-row sums reduce inside the lane.  W_K
// fragments stream from the fragment-tiled copy (wtile_off) into a ring of
// registers (the k loop has no barriers); wave w owns, in column tile ct, the
// pairs 128 ct + 32 w + [0, 32) (both RoPE members, dc/2 apart) for all BM
// candidates, so no W_K fragment is loaded twice by a workgroup.
#pragma once
#include "common.hpp"

namespace still {

struct RefineKArgs {
  const void* K;          // [H][N][d] RoPE'd keys (IT)
  const void* V;          // [H][N][d] values (IT)
  const double* pos;      // [N] key positions
  const double* invf_b;   // [d/2] base RoPE frequencies (fp64)
  const double* invf_c;   // [dc/2] compactor RoPE frequencies (fp64)
  const f16* wkt;         // W_K fragment-tiled (wtile_off), nc*dc rows x 2d columns
  const void* bias;       // [nc*dc] b_K (TBias) or NULL
  const int* ridx;        // [H*nc][t*R] key of each candidate slot (< 0: empty)
  const int* crow;        // [H*nc][t*R] compacted list: row -> slot
  const int* count;       // [H*nc] rows in each list
  const float* qex;       // [H][t][nc*dc] fp32 q~
  float2* rpart;          // [H*nc][t*R] (dot, sum of squares) per slot
  const float* hscale;    // [H] fp16 range scale of each KV head's rows (applied to the rows and b_K), or NULL
  long N;
  int t, R, H, nc, dc;
  int ntile;              // row tiles per list the grid covers (ntile * H * nc workgroups, looping)
};

// four consecutive I/O values as floats (8-byte load for bf16)
template <class IT> __device__ __forceinline__ void load4f(const IT* p, float* o) {
#pragma unroll
  for (int u = 0; u < 4; ++u) o[u] = to_f32(p[u]);
}
template <> __device__ __forceinline__ void load4f<bf16>(const bf16* p, float* o) {
  const uint2 u = *(const uint2*)p;
  o[0] = __uint_as_float(u.x << 16);
  o[1] = __uint_as_float(u.x & 0xffff0000u);
  o[2] = __uint_as_float(u.y << 16);
  o[3] = __uint_as_float(u.y & 0xffff0000u);
}

// D: base head width d.  BM: candidate rows per workgroup.
template <int D, int BM, class IT, class TBias>
__global__ __launch_bounds__(256) void refine_kernel(RefineKArgs a) {
  constexpr int W = 3 * D;               // contraction width [K_hi | V | K_lo]
  constexpr int KW = 2 * D / 16;         // k steps of W_K's 2d columns
  constexpr int KH = D / 16;             // key steps: K_hi and K_lo use the same W_K fragments
  constexpr int TC = BM / 32;            // candidate tiles (MFMA columns)
  constexpr int PT = 128;                // pairs per column tile (32 per wave)
  constexpr int LA = W + 8;              // LDS row stride (halfs)
  constexpr int RB = KW > 8 ? 8 : 4;     // W_K ring depth (k steps)
  constexpr int HD = D / 2;
  static_assert(KW > RB && KW % RB == 0, "ring slots must repeat across column tiles");
  __shared__ __attribute__((aligned(16))) f16 As[BM * LA];
  __shared__ int2 rinfo[BM];             // (key, latent) of each row
  __shared__ float2 red[4][BM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  // Workgroup ids are dealt to the 8 XCDs round robin; XCD x takes the x-th
  // eighth of the (cross head, KV head, row tile) sequence, so the workgroups
  // of one XCD share few cross heads and their W_K stays in its L2.
  const int T = gridDim.x;
  int q = blockIdx.x;
  if ((T & 7) == 0) q = (q & 7) * (T >> 3) + (q >> 3);
  const int rt0 = q % a.ntile, q2 = q / a.ntile;
  const int h = q2 % a.H, c = q2 / a.H;
  const int b = h * a.nc + c;                     // list (h, c)
  const int cnt = a.count[b];                     // uniform
  const int TR = a.t * a.R;
  const int hh = a.dc >> 1;
  const float hsc = a.hscale ? a.hscale[h] : 1.f;
  const long Ec = (long)a.nc * a.dc;
  const int* crow = a.crow + (long)b * TR;
  const int* ridx = a.ridx + (long)b * TR;

  // The grid covers ntile row tiles of each list; a workgroup takes tiles
  // rt0, rt0 + ntile, ... while they hold rows.
  for (int rt = rt0; rt * BM < cnt; rt += a.ntile) {
    const int r0 = rt * BM;
    __syncthreads();   // the previous tile's LDS reads are done
    // ---- gather: row r of the tile = list row r0 + r (zero past the count)
    for (int r = tid; r < BM; r += 256) {
      int key = 0, lat = 0;
      if (r0 + r < cnt) {
        const int slot = crow[r0 + r];
        key = max(ridx[slot], 0);
        lat = slot / a.R;
      }
      rinfo[r] = make_int2(key, lat);
    }
    __syncthreads();
    const IT* Kh = (const IT*)a.K + (long)h * a.N * D;
    const IT* Vh = (const IT*)a.V + (long)h * a.N * D;
    for (int v = tid; v < BM * (HD / 4); v += 256) {
      const int r = v / (HD / 4), j = (v - r * (HD / 4)) * 4;   // pairs j .. j + 3
      const bool ok = r0 + r < cnt;
      const long n = rinfo[r].x;
      f16* row = As + r * LA;
      float k0[4], k1[4], v0[4], v1[4];
      float cc[4] = {1.f, 1.f, 1.f, 1.f}, ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < 4; ++u) k0[u] = k1[u] = v0[u] = v1[u] = 0.f;
      if (ok) {
        const IT* kr = Kh + n * D;
        const IT* vr = Vh + n * D;
        load4f(kr + j, k0);
        load4f(kr + j + HD, k1);
        load4f(vr + j, v0);
        load4f(vr + j + HD, v1);
        const double pn = a.pos[n];
#pragma unroll
        for (int u = 0; u < 4; ++u) {   // base RoPE of pairs j .. j + 3 at the key's position
          const float2 cs = rope_cs(pn, a.invf_b[j + u]);
          cc[u] = cs.x;
          ss[u] = cs.y;
        }
      }
      half4 h0, h1, l0, l1, w0, w1;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // un-rotation of the base RoPE (rotate-half pairs j, j + d/2), then
        // the head's fp16 range scale
        const float y0 = (k0[u] * cc[u] + k1[u] * ss[u]) * hsc;
        const float y1 = (k1[u] * cc[u] - k0[u] * ss[u]) * hsc;
        h0[u] = (f16)y0;
        h1[u] = (f16)y1;
        l0[u] = (f16)(y0 - (float)h0[u]);
        l1[u] = (f16)(y1 - (float)h1[u]);
        w0[u] = (f16)(v0[u] * hsc);
        w1[u] = (f16)(v1[u] * hsc);
      }
      *(half4*)&row[j] = h0;
      *(half4*)&row[j + HD] = h1;
      *(half4*)&row[D + j] = w0;
      *(half4*)&row[D + j + HD] = w1;
      *(half4*)&row[2 * D + j] = l0;
      *(half4*)&row[2 * D + j + HD] = l1;
    }
    __syncthreads();

    // ---- W_K fragments: member m (0: widths p, 1: widths p + dc/2) of this
    // wave's 32 pairs in column tile ct, k step s
    const f16* wkc = a.wkt + (long)c * a.dc * (2 * D);
    const int nct = (hh + PT - 1) / PT;
    // First pair of this wave's 32 in column tile ct.  A wave with no pairs
    // left there (32 w >= dc/2 in the last tile, e.g. every tile when
    // dc/2 < PT) loads the head's first 32 pairs instead, so every W_K row it
    // reads lies inside the head, and its results are dropped.
    auto ct_ld = [&](int ct) { return (PT * ct + 32 * w < hh) ? PT * ct + 32 * w : 0; };
    auto load_b = [&](int pbase, int m, int s) -> half8 {
      const int row0 = pbase + m * hh;   // multiple of 32, row0 + 31 < dc
      return *(const half8*)(wkc + ((((long)(row0 >> 5) * KW + s) << 9) + 8 * lane));
    };

    float dps[TC], sps[TC];
#pragma unroll
    for (int i = 0; i < TC; ++i) dps[i] = sps[i] = 0.f;

    half8 br[RB][2];
#pragma unroll
    for (int s = 0; s < RB; ++s)
#pragma unroll
      for (int m = 0; m < 2; ++m) br[s][m] = load_b(ct_ld(0), m, s);

    const f16* Ab = As + l32 * LA + 8 * g;
    const TBias* bb = a.bias ? (const TBias*)a.bias + (long)c * a.dc : nullptr;
    const float* qh = a.qex + (long)h * a.t * Ec + (long)c * a.dc;
    for (int ct = 0; ct < nct; ++ct) {
      const int ctn = ct_ld(ct + 1 < nct ? ct + 1 : ct);
      f32x16 acc[TC][2];
#pragma unroll
      for (int i = 0; i < TC; ++i) acc[i][0] = acc[i][1] = zero16();
      // step s < KH: [K_hi | K_lo] columns s of the rows against W_K's key
      // step s (one W_K fragment, two products); s >= KH: the V columns
      half8 af[2][TC], al[2][TC];
#pragma unroll
      for (int i = 0; i < TC; ++i) {
        af[0][i] = *(const half8*)&Ab[32 * i * LA];
        al[0][i] = *(const half8*)&Ab[32 * i * LA + 2 * D];
      }
#pragma unroll
      for (int s = 0; s < KW; ++s) {
        if (s + 1 < KW) {
#pragma unroll
          for (int i = 0; i < TC; ++i) {
            af[(s + 1) & 1][i] = *(const half8*)&Ab[32 * i * LA + 16 * (s + 1)];
            if (s + 1 < KH) al[(s + 1) & 1][i] = *(const half8*)&Ab[32 * i * LA + 2 * D + 16 * (s + 1)];
          }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < TC; ++i)
#pragma unroll
          for (int m = 0; m < 2; ++m) {
            acc[i][m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(br[s % RB][m], af[s & 1][i], acc[i][m], 0, 0, 0);
            if (s < KH)
              acc[i][m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(br[s % RB][m], al[s & 1][i], acc[i][m], 0, 0, 0);
          }
        // refill the ring slot with step s + RB (of the next column tile past the end)
        const int sn = s + RB;
#pragma unroll
        for (int m = 0; m < 2; ++m) br[s % RB][m] = sn < KW ? load_b(ct_ld(ct), m, sn) : load_b(ctn, m, sn - KW);
        __builtin_amdgcn_sched_barrier(0);
      }

      // ---- epilogue of the column tile: lane holds candidate 32 i + l32 and
      // pairs p0 + 8 jq + [0, 4) (register j = 4 jq + u)
      const int p0 = PT * ct + 32 * w + 4 * g;
      if (PT * ct + 32 * w < hh) {
        float bs0[16], bs1[16];
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          float t0[4] = {0.f, 0.f, 0.f, 0.f}, t1[4] = {0.f, 0.f, 0.f, 0.f};
          if (bb) {
            load4f(bb + p0 + 8 * jq, t0);
            load4f(bb + p0 + 8 * jq + hh, t1);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            bs0[4 * jq + u] = t0[u] * hsc;
            bs1[4 * jq + u] = t1[u] * hsc;
          }
        }
#pragma unroll
        for (int i = 0; i < TC; ++i) {
          const int2 ri = rinfo[32 * i + l32];
          const double pk = a.pos[ri.x];
          const float* qr = qh + (long)ri.y * Ec + p0;
          float dp = 0.f, sp = 0.f;
#pragma unroll
          for (int jq = 0; jq < 4; ++jq) {
            // four rotations at a time (keeps the fp64 angle work from being
            // hoisted all at once, which would cost occupancy)
            __builtin_amdgcn_sched_barrier(0);
            const f32x4 q0 = *(const f32x4*)(qr + 8 * jq);
            const f32x4 q1 = *(const f32x4*)(qr + 8 * jq + hh);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const float2 rc = rope_cs(pk, a.invf_c[p0 + 8 * jq + u]);
              const float v0 = acc[i][0][4 * jq + u] + bs0[4 * jq + u];
              const float v1 = acc[i][1][4 * jq + u] + bs1[4 * jq + u];
              sp += v0 * v0 + v1 * v1;
              const float y0 = v0 * rc.x - v1 * rc.y, y1 = v1 * rc.x + v0 * rc.y;
              dp += y0 * q0[u] + y1 * q1[u];
            }
          }
          dps[i] += dp;
          sps[i] += sp;
        }
      }
    }

    // ---- per-row sums: the two lane halves, then the 4 waves
#pragma unroll
    for (int i = 0; i < TC; ++i) {
      const float dp = dps[i] + __shfl_xor(dps[i], 32);
      const float sp = sps[i] + __shfl_xor(sps[i], 32);
      if (g == 0) red[w][32 * i + l32] = make_float2(dp, sp);
    }
    __syncthreads();
    for (int r = tid; r < BM; r += 256) {
      if (r0 + r >= cnt) continue;
      float2 s = red[0][r];
#pragma unroll
      for (int u = 1; u < 4; ++u) {
        s.x += red[u][r].x;
        s.y += red[u][r].y;
      }
      a.rpart[(long)b * TR + crow[r0 + r]] = s;
    }
  }
}

}  // namespace still
