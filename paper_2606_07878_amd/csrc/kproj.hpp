// kproj.hpp - cross-attention key projection of the fp16 path, fused with
// what follows it: k~ = X W_K^T + b_K for every cross head, the per-head sum
// of squares of k~ (QK-norm), the compactor RoPE at the key positions and the
// store in the fragment-tiled key layout read by the cross-attention kernel.
//
// The product is computed transposed, k~^T = W_K X^T: MFMA rows are widths
// (W_K rows, A operand) and columns are keys (X rows, B operand).  Then lane l
// of a 32x32 accumulator holds key l % 32 and widths 8 (j / 4) + 4 g + j % 4
// (g = l / 32, register j), and the RoPE partner of width x (x + dc/2) sits in
// the same register of the accumulator of the width tile dc/2 further on.
// Bias, sum of squares, rotation and the fp16 conversion all happen in
// registers; registers 8 s .. 8 s + 7 of a lane are one 16-byte unit of the
// tiled key layout (width step s of the tile, lane slot l), so every store is
// a coalesced 1 KB per wave.  Within a width step of 16 the layout holds, in
// lane half g, widths {4g .. 4g+3, 8+4g .. 8+4g+3} (kperm_width); the query
// projection writes q in the same order, so the cross-attention pairs every
// width of q with the same width of k.
//
// Workgroup = KPW key positions x all H KV heads (128 rows, KPW = 128 / H),
// 4 waves.  The X rows stay in LDS for the whole workgroup; the rotation
// table rows of the KPW positions are staged in LDS per tile of 32 pairs and
// shared by all cross heads and KV heads, and so are the tile's b_K values
// (the epilogue then has no global loads to wait for: on gfx9 such a wait
// also waits for the wave's earlier key stores).  Wave w takes the cross heads
// c = w, w + 4, ...; W_K comes from a fragment-tiled fp16 copy (wtile_off).
#pragma once
#include "common.hpp"

namespace still {

// Fragment-tiled W (rows = output widths, contiguous input dimension d2):
// [row / 32][col / 16][lane = row % 32 + 32 * ((col / 8) % 2)][col % 8]
__host__ __device__ __forceinline__ long wtile_off(long row, long col, long d2) {
  return (((row >> 5) * (d2 >> 4) + (col >> 4)) << 9) + (((row & 31) + (((col >> 3) & 1) << 5)) << 3) + (col & 7);
}

// Width held by position p (0..15) of a 16-width step in the permuted order.
__host__ __device__ __forceinline__ int kperm_width(int p) {
  const int g = p >> 3, e = p & 7;
  return e < 4 ? 4 * g + e : 8 + 4 * g + (e - 4);
}

// W (fp16, row-major [rows][d2]) -> fragment-tiled copy; one thread per
// 16-byte unit.
static __global__ void tile_w_kernel(const f16* __restrict__ w, long rows, int d2, f16* __restrict__ out) {
  const long units = rows * (d2 / 8);
  for (long u = blockIdx.x * (long)blockDim.x + threadIdx.x; u < units; u += (long)gridDim.x * blockDim.x) {
    const long row = u / (d2 / 8);
    const int col = (int)(u - row * (d2 / 8)) * 8;
    *(uint4*)(out + wtile_off(row, col, d2)) = *(const uint4*)(w + row * d2 + col);
  }
}

struct KprojArgs {
  const f16* X;         // [H*N][d2] RoPE-fixed keys and values
  const f16* wkt;       // W_K fragment-tiled (wtile_off), nc*dc rows
  const void* bias;     // [nc*dc] b_K (TBias) or NULL
  const double* pos;    // [N] key positions
  const double* invf;   // [dc/2] compactor RoPE frequencies (fp64)
  f16* k;               // tiled keys (ktile_off with npad keys per head), permuted widths
  float* part;          // [nc][H*N] sum of squares of k~ (one partial per row and cross head)
  const float* hscale;  // [H] fp16 range scale of the staged X of each KV head (the bias is scaled with it), or NULL
  int H, N, nc, dc, kpw;
  long npad;
};

// TPW: capacity of the table stage in key positions (a.kpw <= TPW).
template <int D2, int TPW, class TBias>
__global__ __launch_bounds__(256, 2) void kproj_kernel(KprojArgs a) {
  constexpr int LX = D2 + 8;          // X row stride in LDS (halfs)
  constexpr int KS = D2 / 16;         // k steps
  constexpr int RING = 2;             // W_K fragment prefetch depth (k steps)
  static_assert(KS % RING == 0, "k steps");
  __shared__ __attribute__((aligned(16))) f16 Xs[128 * LX];
  // table stage rows of 32 (cos, sin) pairs, padded to 34 so that the lanes
  // of a wave reading the same pairs of different key positions hit
  // different LDS banks (a 256-byte stride maps every row to one bank group)
  constexpr int TS = 34;
  __shared__ __attribute__((aligned(16))) float2 Ts[2 * TPW * TS];
  // bias stage: per buffer, the 8 cross heads 4 cb .. 4 cb + 7 of the current
  // pair round, widths 32 p .. 32 p + 31 of each RoPE half (4 values per uint2)
  __shared__ uint2 Bs[2][8][16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const int kpw = a.kpw;
  const int n0 = blockIdx.x * kpw;
  const long HN = (long)a.H * a.N;
  const int hh = a.dc >> 1;
  const int NPT = a.dc / 64;          // tiles of 32 pairs per cross head

  // ---- X rows of the workgroup into LDS (rows of absent heads/keys: zero)
  for (int v = tid; v < 128 * (D2 / 8); v += 256) {
    const int r = v / (D2 / 8), col = (v - r * (D2 / 8)) * 8;
    const int h = r / kpw, n = n0 + (r - h * kpw);
    uint4 val = make_uint4(0, 0, 0, 0);
    if (h < a.H && n < a.N) val = *(const uint4*)(a.X + ((long)h * a.N + n) * D2 + col);
    *(uint4*)&Xs[r * LX + col] = val;
  }
  // rotation tile: (cos, sin) of key positions n0 .. n0 + kpw - 1 for pairs
  // 32p .. 32p + 31, computed from the fp64 positions and frequencies
  const TBias* bias = (const TBias*)a.bias;
  auto load_tab = [&](int p, int buf, int cbv) {
    if (tid < 128) {
      const int lc = tid >> 4, u = tid & 15, c = 4 * cbv + lc;
      uint2 val = make_uint2(0, 0);
      if (bias && c < a.nc)
        val = *(const uint2*)(bias + (long)c * a.dc + (u < 8 ? 32 * p + 4 * u : hh + 32 * p + 4 * (u - 8)));
      Bs[buf][lc][u] = val;
    }
    for (int v = tid; v < kpw * 16; v += 256) {
      const int pos = v >> 4, j2 = (v & 15) * 2;
      const int n = n0 + pos;
      f32x4 cs = {1.f, 0.f, 1.f, 0.f};
      if (n < a.N) {
        const double pn = a.pos[n];
        const float2 c0 = rope_cs(pn, a.invf[32 * p + j2]), c1 = rope_cs(pn, a.invf[32 * p + j2 + 1]);
        cs = f32x4{c0.x, c0.y, c1.x, c1.y};
      }
      *(f32x4*)&Ts[(buf * kpw + pos) * TS + j2] = cs;
    }
  };
  load_tab(0, 0, 0);

  // this lane's key in each key tile: row, KV head, key index
  int kh[4], kn[4];
  bool kok[4];
  float bsc[4];   // bias scale of the key's KV head
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const int r = 32 * kt + l32;
    kh[kt] = r / kpw;
    kn[kt] = n0 + (r - kh[kt] * kpw);
    kok[kt] = kh[kt] < a.H && kn[kt] < a.N;
    bsc[kt] = (a.hscale && kh[kt] < a.H) ? a.hscale[kh[kt]] : 1.f;
  }
  // Every wave runs the same loop trip counts (the barriers are workgroup
  // wide); wave w computes cross heads w + 4 (cb + i) that exist.
  const int rounds = (a.nc + 3) / 4;    // cross heads per wave, at most
  float ss0[4], ss1[4];                 // per key tile, for the two cross heads of a pair
  auto flush_ss = [&](int c, float (&ss)[4]) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const float tot = ss[kt] + __shfl_xor(ss[kt], 32);
      if (g == 0 && kok[kt]) a.part[(long)c * HN + (long)kh[kt] * a.N + kn[kt]] = tot;
      ss[kt] = 0.f;
    }
  };

  int tb = 0;   // table buffer of the current tile
  for (int cb = 0; cb < rounds; cb += 2) {   // pairs of this wave's cross heads
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) ss0[kt] = ss1[kt] = 0.f;
    for (int p = 0; p < NPT; ++p) {
      __syncthreads();                       // X rows / table tile p visible; the other buffer free
      if (p + 1 < NPT) load_tab(p + 1, tb ^ 1, cb);
      else if (cb + 2 < rounds) load_tab(0, tb ^ 1, cb + 2);   // the next pair of cross heads restarts at tile 0
      const float2* T = Ts + (size_t)tb * kpw * TS;
#pragma unroll 1
      for (int i = 0; i < 2; ++i) {
        const int c = w + 4 * (cb + i);
        if (c < a.nc) {
        // width tiles (32 rows of W_K) of the low and high RoPE halves
        const long wt_lo = ((long)c * a.dc + 32 * p) >> 5, wt_hi = wt_lo + (hh >> 5);
        const f16* alo = a.wkt + (wt_lo * KS << 9) + 8 * lane;
        const f16* ahi = a.wkt + (wt_hi * KS << 9) + 8 * lane;
        f32x16 acc[2][4];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) acc[hf][kt] = zero16();
        half8 ra[RING][2];
#pragma unroll
        for (int s = 0; s < RING; ++s) {
          ra[s][0] = *(const half8*)(alo + (s << 9));
          ra[s][1] = *(const half8*)(ahi + (s << 9));
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          half8 b[4];
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) b[kt] = *(const half8*)&Xs[(32 * kt + l32) * LX + 16 * ks + 8 * g];
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) {
            acc[0][kt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ra[ks % RING][0], b[kt], acc[0][kt], 0, 0, 0);
            acc[1][kt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ra[ks % RING][1], b[kt], acc[1][kt], 0, 0, 0);
          }
          if (ks + RING < KS) {
            ra[ks % RING][0] = *(const half8*)(alo + ((ks + RING) << 9));
            ra[ks % RING][1] = *(const half8*)(ahi + ((ks + RING) << 9));
          }
        }
        // ---- epilogue: bias, sum of squares, rotation, fp16, tiled stores
        // biases of this lane's widths: 4 consecutive values per group q (8-byte loads)
        static_assert(sizeof(TBias) == 2, "2-byte bias type");
        uint2 bl[4], bu[4];
        {
          const uint2* bsrc = &Bs[tb][c - 4 * cb][0];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            bl[q] = bsrc[2 * q + g];
            bu[q] = bsrc[8 + 2 * q + g];
          }
        }
        auto bias_at = [&](const uint2& v, int u) -> float {
          const uint32_t wd = u < 2 ? v.x : v.y;
          const TBias e = __builtin_bit_cast(TBias, (uint16_t)((u & 1) ? (wd >> 16) : (wd & 0xffffu)));
          return to_f32(e);
        };
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const int pos = kn[kt] - n0;
          const float2* tr = T + (kok[kt] ? pos : 0) * TS;
          half8 olo[2], ohi[2];
          float ss = 0.f;
#pragma unroll
          for (int q = 0; q < 4; ++q) {   // registers 4q .. 4q + 3: pairs 8q + 4g .. 8q + 4g + 3 of the tile
            const f32x4 c01 = *(const f32x4*)&tr[8 * q + 4 * g];
            const f32x4 c23 = *(const f32x4*)&tr[8 * q + 4 * g + 2];
            const float cs[4] = {c01[0], c01[2], c23[0], c23[2]};
            const float sn[4] = {c01[1], c01[3], c23[1], c23[3]};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int j = 4 * q + u;
              const float blo = bias_at(bl[q], u) * bsc[kt], bhi = bias_at(bu[q], u) * bsc[kt];
              const float ylo = acc[0][kt][j] + blo, yhi = acc[1][kt][j] + bhi;
              ss += ylo * ylo + yhi * yhi;
              olo[j >> 3][j & 7] = (f16)(ylo * cs[u] - yhi * sn[u]);
              ohi[j >> 3][j & 7] = (f16)(yhi * cs[u] + ylo * sn[u]);
            }
          }
          if (i == 0) ss0[kt] += ss;
          else ss1[kt] += ss;
          if (kok[kt]) {
            const long hck = (long)kh[kt] * a.nc + c;
#pragma unroll
            for (int s = 0; s < 2; ++s) {   // width steps 2p + s (low half) and (dc/2)/16 + 2p + s (high half)
              const long flo = ((hck * (a.npad >> 5) + (kn[kt] >> 5)) * (a.dc >> 4) + 2 * p + s) << 9;
              const long fhi = flo + ((long)(hh >> 4) << 9);
              const long slot = ((kn[kt] & 31) + 32 * g) * 8;
              // streaming stores: the keys are read back only by the next
              // kernel; W_K and the X rows stay in L2
              __builtin_nontemporal_store(olo[s], (half8*)(a.k + flo + slot));
              __builtin_nontemporal_store(ohi[s], (half8*)(a.k + fhi + slot));
            }
          }
        }
        }
      }
      tb ^= 1;
    }
    if (w + 4 * cb < a.nc) flush_ss(w + 4 * cb, ss0);
    if (w + 4 * (cb + 1) < a.nc) flush_ss(w + 4 * (cb + 1), ss1);
  }
}

}  // namespace still
