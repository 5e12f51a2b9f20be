// Small-batch kernels (R <= 16 rows in a pass: batch x (K+1) <= 16).
// At this size every contraction is a weight stream, so the kernels aim at
// memory-level parallelism and few launches:
//   - a 16-feature strip is split along K over NW waves of one block; each
//     wave issues all of its tile loads before its MFMAs and the partial
//     accumulators are summed in LDS in wave order (deterministic);
//   - RMSNorm is a prologue that recomputes the (few) normalised rows into
//     LDS, which then feeds the MFMA B operand;
//   - the MoE down projection is n-tile-major: the blocks of a 16-feature
//     strip share the touched experts round-robin, and the strip's last
//     block adds the (exact fixed-point) sum straight into the residual
//     stream.
#pragma once
#include "common.h"
#include "kernels_mfma.h"

namespace mtp {

constexpr int SR_MAX = 16;  // rows of the small-batch path
constexpr int XPAD = 8;     // LDS row padding (bf16 elements)

// acc += tiles [t0, t1) of a packed strip against this lane's B row
// (global or LDS).  Batches of BT tiles, double-buffered: the loads of the
// next batch are in flight while the current one is multiplied.  The
// staging costs 4*BT uint4 registers per lane: BT = 8 for 256-thread blocks,
// 4 for 1024-thread blocks (128 VGPRs per lane at most).
template <int BT>
__device__ __forceinline__ void sk_load(const uint4* __restrict__ A, int t, int t1,
                                        const uint16_t* xrow, int koff, uint4 (&a)[BT],
                                        uint4 (&b)[BT], bool nt) {
  const int lane = threadIdx.x & 63;
  const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int u = 0; u < BT; ++u) {
    if (t + u < t1) {
      a[u] = ld_tile(A + (size_t)(t + u) * 64 + lane, nt);
      b[u] = xrow ? ldx(xrow + (t + u) * 32 + koff) : z;
    }
  }
}

template <int BT = 8>
__device__ __forceinline__ f32x4_t sk_range(const uint4* __restrict__ A, int t0, int t1,
                                            const uint16_t* xrow, f32x4_t acc, bool nt = false) {
  const int koff = 8 * ((threadIdx.x & 63) >> 4);
  const uint4 z = make_uint4(0, 0, 0, 0);
  uint4 a[BT], b[BT];
#pragma unroll
  for (int u = 0; u < BT; ++u) a[u] = b[u] = z;  // every staged register defined
  if (t0 < t1) sk_load<BT>(A, t0, t1, xrow, koff, a, b, nt);
  for (int t = t0; t < t1; t += BT) {
    uint4 an[BT], bn[BT];
#pragma unroll
    for (int u = 0; u < BT; ++u) an[u] = bn[u] = z;
    if (t + BT < t1) sk_load<BT>(A, t + BT, t1, xrow, koff, an, bn, nt);
#pragma unroll
    for (int u = 0; u < BT; ++u)
      if (t + u < t1) acc = mfma16(a[u], b[u], acc);
#pragma unroll
    for (int u = 0; u < BT; ++u) {
      a[u] = an[u];
      b[u] = bn[u];
    }
  }
  return acc;
}

// sk_range with the B row in LDS (xl) and the first batch (tiles t0..)
// already loaded into a: only the weight tiles are global loads, so
// waiting on a batch never waits on a B read
template <int BT = 8>
__device__ __forceinline__ f32x4_t sk_range_lx(const uint4* __restrict__ A, int t0, int t1,
                                               const uint16_t* xl, f32x4_t acc, bool nt,
                                               uint4 (&a)[BT]) {
  const int lane = threadIdx.x & 63, koff = 8 * (lane >> 4);
  for (int t = t0; t < t1; t += BT) {
    uint4 an[BT];
#pragma unroll
    for (int u = 0; u < BT; ++u)
      an[u] = t + BT + u < t1 ? ld_tile(A + (size_t)(t + BT + u) * 64 + lane, nt)
                              : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < BT; ++u)
      if (t + u < t1) acc = mfma16(a[u], *(const uint4*)(xl + (t + u) * 32 + koff), acc);
#pragma unroll
    for (int u = 0; u < BT; ++u) a[u] = an[u];
  }
  return acc;
}

// up to MAXT tiles of a strip, loaded into registers ahead of their use
template <int MAXT>
__device__ __forceinline__ void preload(const uint4* __restrict__ A, int t0, int n,
                                        uint4 (&a)[MAXT], bool nt = false) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int u = 0; u < MAXT; ++u)
    a[u] = u < n ? ld_tile(A + (size_t)(t0 + u) * 64 + lane, nt) : make_uint4(0, 0, 0, 0);
}

// acc += preloaded tiles a[0..n) against this lane's B row; the B operands
// are read CH at a time (CH = MAXT: all reads issued first, for a B row in
// global memory; a small CH saves registers when the row is in LDS)
template <int MAXT, int CH = MAXT>
__device__ __forceinline__ f32x4_t mma_pre(const uint4 (&a)[MAXT], int t0, int n,
                                           const uint16_t* xrow, f32x4_t acc) {
  static_assert(MAXT % CH == 0, "chunk must divide the tile count");
  const int koff = 8 * ((threadIdx.x & 63) >> 4);
  const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int c0 = 0; c0 < MAXT; c0 += CH) {
    uint4 b[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u)
      b[u] = (c0 + u < n && xrow) ? ldx(xrow + (t0 + c0 + u) * 32 + koff) : z;
#pragma unroll
    for (int u = 0; u < CH; ++u)
      if (c0 + u < n) acc = mfma16(a[c0 + u], b[u], acc);
  }
  return acc;
}

// two preloaded strips against the same B row (one B read per tile)
template <int MAXT, int CH = MAXT>
__device__ __forceinline__ void mma_pre2(const uint4 (&a1)[MAXT], const uint4 (&a2)[MAXT], int t0,
                                         int n, const uint16_t* xrow, f32x4_t& c1, f32x4_t& c2) {
  static_assert(MAXT % CH == 0, "chunk must divide the tile count");
  const int koff = 8 * ((threadIdx.x & 63) >> 4);
  const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int c0 = 0; c0 < MAXT; c0 += CH) {
    uint4 b[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u)
      b[u] = (c0 + u < n && xrow) ? ldx(xrow + (t0 + c0 + u) * 32 + koff) : z;
#pragma unroll
    for (int u = 0; u < CH; ++u)
      if (c0 + u < n) {
        c1 = mfma16(a1[c0 + u], b[u], c1);
        c2 = mfma16(a2[c0 + u], b[u], c2);
      }
  }
}

// tiles per wave (K / 32 / 4 waves) -> register array size
#define MTP_MAXT_DISPATCH(per, F)      \
  do {                                 \
    if ((per) <= 4) { F(4); }          \
    else if ((per) <= 8) { F(8); }     \
    else if ((per) <= 10) { F(10); }   \
    else { F(16); }                    \
  } while (0)

// sum of the NW per-wave accumulators in wave order; the result is valid
// in wave 0.  red holds NW*64 f32x4.
template <int NW>
__device__ __forceinline__ f32x4_t block_acc_sum(f32x4_t acc, f32x4_t* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  red[w * 64 + lane] = acc;
  __syncthreads();
  f32x4_t s = red[lane];
  if (w == 0) {
#pragma unroll
    for (int x = 1; x < NW; ++x) s += red[x * 64 + lane];
  }
  return s;
}

// RMSNorm of rows r < R of src (row stride H, H % 256 == 0, H <= 256*NV)
// with gain g into LDS xs[r][ldl] (bf16).  Wave w takes rows w, w+nw, ...;
// each row and the gain are loaded together, before the row's reduction,
// so no load waits on a reduction.
// With skip_first, each wave starts at its second row (its first was done
// by norm_row_load / norm_row_store).
template <int NV>
__device__ __forceinline__ void norm_rows_lds(int R, int H, const float* __restrict__ src,
                                              const float* __restrict__ g, float eps,
                                              uint16_t* xs, int ldl, bool skip_first = false) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int n4 = H / 256;  // float4 per lane
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int r = w + (skip_first ? nw : 0); r < R; r += nw) {
    float4 xv[NV], gv[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      xv[u] = u < n4 ? ld_f4(src + (size_t)r * H + (u * 64 + lane) * 4) : z;
      gv[u] = u < n4 ? ld_f4(g + (u * 64 + lane) * 4) : z;
    }
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u)
      ss += xv[u].x * xv[u].x + xv[u].y * xv[u].y + xv[u].z * xv[u].z + xv[u].w * xv[u].w;
    ss = wave_sum(ss);
    const float rinv = rsqrtf(ss / (float)H + eps);
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      if (u < n4) {
        uint2 pk;
        pk.x = (uint32_t)f2bf(xv[u].x * rinv * gv[u].x) |
               ((uint32_t)f2bf(xv[u].y * rinv * gv[u].y) << 16);
        pk.y = (uint32_t)f2bf(xv[u].z * rinv * gv[u].z) |
               ((uint32_t)f2bf(xv[u].w * rinv * gv[u].w) << 16);
        *(uint2*)(xs + r * ldl + (u * 64 + lane) * 4) = pk;
      }
    }
  }
}

// One row of the same RMSNorm held in registers: its loads can be issued
// before a kernel's weight tiles, so the row's sum is formed while the
// tiles are in flight (the result is that of norm_rows_lds).
template <int NV>
struct NormRow {
  float4 x[NV], g[NV];
};
template <int NV>
__device__ __forceinline__ void norm_row_load(int H, const float* __restrict__ src,
                                              const float* __restrict__ g, NormRow<NV>& nr) {
  const int lane = threadIdx.x & 63, n4 = H / 256;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    nr.x[u] = u < n4 ? ld_f4(src + (u * 64 + lane) * 4) : z;
    nr.g[u] = u < n4 ? ld_f4(g + (u * 64 + lane) * 4) : z;
  }
}
template <int NV>
__device__ __forceinline__ void norm_row_store(int H, float eps, const NormRow<NV>& nr,
                                               uint16_t* dst) {
  const int lane = threadIdx.x & 63, n4 = H / 256;
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u)
    ss += nr.x[u].x * nr.x[u].x + nr.x[u].y * nr.x[u].y + nr.x[u].z * nr.x[u].z +
          nr.x[u].w * nr.x[u].w;
  ss = wave_sum(ss);
  const float rinv = rsqrtf(ss / (float)H + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    if (u < n4) {
      uint2 pk;
      pk.x = (uint32_t)f2bf(nr.x[u].x * rinv * nr.g[u].x) |
             ((uint32_t)f2bf(nr.x[u].y * rinv * nr.g[u].y) << 16);
      pk.y = (uint32_t)f2bf(nr.x[u].z * rinv * nr.g[u].z) |
             ((uint32_t)f2bf(nr.x[u].w * rinv * nr.g[u].w) << 16);
      *(uint2*)(dst + (u * 64 + lane) * 4) = pk;
    }
  }
}

// RMSNorm of rows x[idx ? idx[o] : o] (float32, row stride H) with gain
// g, one wave per output row o, every load issued before the sum: float32
// to yf[o*H] and/or bf16 to yb[o*H] (each optional).
template <int NV>
__global__ void __launch_bounds__(64) k_norm_rows(int H, const float* __restrict__ x,
                                                  const int32_t* __restrict__ idx,
                                                  const float* __restrict__ g, float eps,
                                                  float* __restrict__ yf,
                                                  uint16_t* __restrict__ yb) {
  const int o = blockIdx.x, lane = threadIdx.x, n4 = H / 256;
  const int r = idx ? idx[o] : o;
  NormRow<NV> nr;
  norm_row_load<NV>(H, x + (size_t)r * H, g, nr);
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u)
    ss += nr.x[u].x * nr.x[u].x + nr.x[u].y * nr.x[u].y + nr.x[u].z * nr.x[u].z +
          nr.x[u].w * nr.x[u].w;
  ss = wave_sum(ss);
  const float rinv = rsqrtf(ss / (float)H + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    if (u < n4) {
      const float4 y = make_float4(nr.x[u].x * rinv * nr.g[u].x, nr.x[u].y * rinv * nr.g[u].y,
                                   nr.x[u].z * rinv * nr.g[u].z, nr.x[u].w * rinv * nr.g[u].w);
      const int j4 = u * 64 + lane;
      if (yf) ((float4*)(yf + (size_t)o * H))[j4] = y;
      if (yb) {
        uint2 pk;
        pk.x = (uint32_t)f2bf(y.x) | ((uint32_t)f2bf(y.y) << 16);
        pk.y = (uint32_t)f2bf(y.z) | ((uint32_t)f2bf(y.w) << 16);
        ((uint2*)(yb + (size_t)o * H))[j4] = pk;
      }
    }
  }
}

// float4 per lane of a row for the register tile count MAXT (= H/128
// rounded up): H/256 <= (MAXT+1)/2
#define MTP_NV(MAXT) (((MAXT) + 1) / 2)

// ---------------------------------------------------------------- dense split-K
// Y[r][n] (=|+=) X[r] . W[n], one 16-feature strip (blockIdx.x) x one
// 16-row group (blockIdx.y) per block, K split over NW waves.  X bf16 rows
// in global memory.  MAXT > 0: each wave's per = nkt/NW <= MAXT tiles are
// all loaded first (and the residual being added to, by wave 0), so the
// block waits on one round of loads; MAXT == 0 streams the tiles in
// double-buffered batches (long K).
template <int NW, bool ADD, int MAXT>
__global__ void __launch_bounds__(NW * 64) k_s_mm(int R, int N, int nkt,
                                                  const uint16_t* __restrict__ X, int ldx_,
                                                  const uint4* __restrict__ Wp,
                                                  float* __restrict__ Y, int ldy) {
  __shared__ f32x4_t red[NW * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nt = blockIdx.x;
  const int r = blockIdx.y * 16 + (lane & 15);  // 16-row group blockIdx.y
  const uint16_t* xrow = r < R ? X + (size_t)r * ldx_ : nullptr;
  const int per = nkt / NW;
  const int n = nt * 16 + 4 * (lane >> 4);
  const bool out = w == 0 && r < R && n < N;
  f32x4_t acc;
  float4 y0 = make_float4(0.f, 0.f, 0.f, 0.f);
  if constexpr (MAXT > 0) {
    uint4 a[MAXT];
    preload<MAXT>(Wp + (size_t)nt * nkt * 64, w * per, per, a, gridDim.y == 1);
    if (ADD && out) y0 = ld_f4(Y + (size_t)r * ldy + n);
    acc = mma_pre<MAXT, (NW >= 16 && MAXT > 8) ? MAXT / 2 : MAXT>(a, w * per, per, xrow,
                                                                  f32x4_t{0.f, 0.f, 0.f, 0.f});
  } else {
    if (ADD && out) y0 = ld_f4(Y + (size_t)r * ldy + n);
    acc = sk_range<(NW >= 16 ? 4 : 8)>(Wp + (size_t)nt * nkt * 64, w * per, (w + 1) * per, xrow,
                                        f32x4_t{0.f, 0.f, 0.f, 0.f}, gridDim.y == 1);
  }
  acc = block_acc_sum<NW>(acc, red);
  if (!out) return;
  *(float4*)(Y + (size_t)r * ldy + n) =
      make_float4(acc[0] + y0.x, acc[1] + y0.y, acc[2] + y0.z, acc[3] + y0.w);
}

// ---------------------------------------------------------------- QKV
// Task = blockIdx.x: a q/k rotate-half pair of strips (RoPE in registers)
// or a v strip; rows = 16-row group blockIdx.y; K split over 4 waves (<= 16
// tiles each).  Each wave first issues its weight-tile loads, then the
// block computes x = RMSNorm(h; g) of its rows into LDS (the prologue
// overlaps the weight fetch) -- or, with xg, reads normalised bf16 rows.
// q -> q_out (float32), k/v -> cache at the row position.
template <int MAXT, bool EARLY = false>
__global__ void __launch_bounds__(256) k_s_qkv(int R, int C, int H, int nh, int dh,
                                               const float* __restrict__ h,
                                               const float* __restrict__ g, float eps,
                                               const uint16_t* __restrict__ xg,
                                               const uint4* __restrict__ Wp,
                                               const float2* __restrict__ rope,
                                               const int32_t* __restrict__ row_pos,
                                               const int32_t* __restrict__ row_valid,
                                               uint16_t* __restrict__ cache, size_t seq_stride,
                                               int cap, float* __restrict__ q_out) {
  extern __shared__ __align__(16) uint16_t xs[];  // [R][H + XPAD]
  __shared__ f32x4_t red[2 * 4 * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ldl = H + XPAD, nkt = H / 32, per = nkt / 4;
  const int D = nh * dh, half = dh / 2, tph = dh / 32;
  const int task = blockIdx.x, n_pair = 2 * nh * tph;
  const bool pair = task < n_pair;
  int sec = 0, hh = 0, pt = 0, ta, tb;
  if (pair) {
    sec = task / (nh * tph);
    const int rest = task % (nh * tph);
    hh = rest / tph;
    pt = rest % tph;
    ta = (sec * D + hh * dh) / 16 + pt;
    tb = ta + tph;
  } else {
    ta = 2 * D / 16 + (task - n_pair);
    tb = ta;
  }
  constexpr int NV = MTP_NV(MAXT);
  const int r0 = blockIdx.y * 16;
  const int nloc = min(16, R - r0);
  // EARLY (prologue mode): each wave's first row is loaded ahead of the
  // weight tiles and normalised while they are in flight
  NormRow<NV> nr0;
  const bool early = EARLY && !xg && w < nloc;
  if (early) norm_row_load<NV>(H, h + (size_t)(r0 + w) * H, g, nr0);
  uint4 a0[MAXT], a1[MAXT];
  const bool once = gridDim.y == 1;  // one row group: every tile is read once
  preload<MAXT>(Wp + (size_t)ta * nkt * 64, w * per, per, a0, once);
  preload<MAXT>(Wp + (size_t)tb * nkt * 64, w * per, pair ? per : 0, a1, once);
  // row bookkeeping and the RoPE factors of this lane's features, loaded
  // before the prologue so none of them waits on a reduction
  const int r = r0 + (lane & 15);
  const int valid = r < R ? row_valid[r] : 0;
  const int pos = r < R ? row_pos[r] : 0;
  float2 cs[4] = {};
  if (pair && w == 0 && r < R) {
    const int p = valid ? pos : 0;
#pragma unroll
    for (int t = 0; t < 4; ++t) cs[t] = rope[(size_t)p * half + pt * 16 + 4 * (lane >> 4) + t];
  }
  // B rows from global memory (xg) or LDS (prologue): two call sites, so
  // each reads with its own load instruction rather than a generic one
  const f32x4_t z4 = {0.f, 0.f, 0.f, 0.f};
  f32x4_t c0 = z4, c1 = z4;
  if (xg) {
    const uint16_t* xrow = r < R ? xg + (size_t)r * H : nullptr;
    if (pair) mma_pre2<MAXT, (MAXT % 2 == 0 ? MAXT / 2 : MAXT)>(a0, a1, w * per, per, xrow, c0, c1);
    else c0 = mma_pre<MAXT>(a0, w * per, per, xrow, z4);
  } else {
    if (early) norm_row_store<NV>(H, eps, nr0, xs + w * ldl);
    norm_rows_lds<NV>(nloc, H, h + (size_t)r0 * H, g, eps, xs, ldl, EARLY);
    __syncthreads();
    // lanes of rows past R read row (lane & 15) of the tile; their columns
    // are not stored
    const uint16_t* xrow = xs + (lane & 15) * ldl;
    if (pair) mma_pre2<MAXT, (MAXT % 2 == 0 ? MAXT / 2 : MAXT)>(a0, a1, w * per, per, xrow, c0, c1);
    else c0 = mma_pre<MAXT>(a0, w * per, per, xrow, z4);
  }
  c0 = block_acc_sum<4>(c0, red);
  if (pair) {
    c1 = block_acc_sum<4>(c1, red + 4 * 64);
    if (w != 0 || r >= R) return;
    const int p = valid ? pos : 0;
    const int b = r / C;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = pt * 16 + 4 * (lane >> 4) + t;
      const float x0 = c0[t], x1 = c1[t];
      const float y0 = x0 * cs[t].x - x1 * cs[t].y, y1 = x1 * cs[t].x + x0 * cs[t].y;
      if (sec == 0) {
        q_out[(size_t)r * D + hh * dh + i] = y0;
        q_out[(size_t)r * D + hh * dh + i + half] = y1;
      } else if (valid) {
        uint16_t* kc = cache + (size_t)b * seq_stride + ((size_t)hh * cap + p) * dh;
        kc[i] = f2bf(y0);
        kc[i + half] = f2bf(y1);
      }
    }
  } else {
    if (w != 0 || r >= R || !valid) return;
    const int b = r / C;
    const int f = (ta - 2 * D / 16) * 16 + 4 * (lane >> 4);
    const int hv = f / dh, d = f % dh;
    uint16_t* vc = cache + (size_t)b * seq_stride + ((size_t)(nh + hv) * cap + pos) * dh + d;
    uint2 pk;
    pk.x = (uint32_t)f2bf(c0[0]) | ((uint32_t)f2bf(c0[1]) << 16);
    pk.y = (uint32_t)f2bf(c0[2]) | ((uint32_t)f2bf(c0[3]) << 16);
    *(uint2*)vc = pk;
  }
}

// ---------------------------------------------------------------- attention
// One 64-key tile of K and V into registers: 16-byte chunk c = threadIdx.x
// + 256u is key c / (DH/8), part c % (DH/8); keys past the capacity clamp
// to the last row (their scores are masked).  A launch reads each cached
// row once, so the loads are non-temporal.
template <int DH, int VPT>
__device__ __forceinline__ void attn_load_tile(const uint16_t* __restrict__ Kc,
                                               const uint16_t* __restrict__ Vc, int t0, int cap,
                                               uint4 (&kr)[VPT], uint4 (&vr)[VPT]) {
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int c = threadIdx.x + 256 * u;
    const int j = min(t0 + c / (DH / 8), cap - 1);
    kr[u] = ld_tile((const uint4*)(Kc + (size_t)j * DH + (c % (DH / 8)) * 8), true);
    vr[u] = ld_tile((const uint4*)(Vc + (size_t)j * DH + (c % (DH / 8)) * 8), true);
  }
}

// Merge of one (row, head)'s n split partials by one wave (n <= 64): lane y
// holds split y's (m, l); the weights e^{m_y - M} go through the wave's LDS
// row w, and each lane sums its dims over the splits with all loads in
// flight.  Writes the bf16 row (zeros for an invalid row or an empty sum).
// The first PRE splits' vectors are loaded with the (m, l) pairs, so their
// sum does not wait on a second round of loads.
template <int DH, int PRE = 16>
__device__ __forceinline__ void attn_merge_row(const float* __restrict__ pp, int n, bool valid,
                                               float* w, uint16_t* __restrict__ out) {
  constexpr int DPL = DH / 64;
  const int lane = threadIdx.x & 63;
  float ov0[PRE][DPL];
#pragma unroll
  for (int u = 0; u < PRE; ++u)
#pragma unroll
    for (int d = 0; d < DPL; ++d)
      ov0[u][d] = u < n ? ld_agent(pp + u * (DH + 2) + lane * DPL + d) : 0.f;
  const float my = lane < n ? ld_agent(pp + lane * (DH + 2) + DH) : -INFINITY;
  const float ly = lane < n ? ld_agent(pp + lane * (DH + 2) + DH + 1) : 0.f;
  const float M = wave_max(my);
  const float fy = (my == -INFINITY) ? 0.f : __expf(my - M);
  const float L = wave_sum(ly * fy);
  w[lane] = fy;
  __builtin_amdgcn_wave_barrier();
  float O[DPL];
#pragma unroll
  for (int d = 0; d < DPL; ++d) O[d] = 0.f;
#pragma unroll
  for (int u = 0; u < PRE; ++u) {
    const float f = u < n ? w[u] : 0.f;
#pragma unroll
    for (int d = 0; d < DPL; ++d) O[d] += ov0[u][d] * f;
  }
  for (int y0 = PRE; y0 < n; y0 += 8) {
    float ov[8][DPL];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int d = 0; d < DPL; ++d)
        ov[u][d] = (y0 + u < n) ? ld_agent(pp + (y0 + u) * (DH + 2) + lane * DPL + d) : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float f = (y0 + u < n) ? w[y0 + u] : 0.f;
#pragma unroll
      for (int d = 0; d < DPL; ++d) O[d] += ov[u][d] * f;
    }
  }
  __builtin_amdgcn_wave_barrier();
  const bool ok = valid && L > 0.f;
#pragma unroll
  for (int d = 0; d < DPL; ++d) out[lane * DPL + d] = f2bf(ok ? O[d] / L : 0.f);
}

// Split-K decode attention, merge fused.  Block (split s, head h,
// z = b*ngroups + g) covers keys [s*spl, (s+1)*spl) of sequence b for the
// NR query rows of group g.  Per 64-key tile the block loads K and V with
// coalesced 16-byte loads (the next tile's loads are issued before the
// current tile is used) into LDS; wave w owns rows w, w+4: lane = key for
// the scores, lane = 2 (or 1) dims for P.V.  Float32 scores and softmax.
// The last block of a (z, head) merges the splits that hold keys and writes
// bf16.
template <int DH, int NR>
__global__ void __launch_bounds__(256) k_s_attn(int C, int nh, int n_split, int spl,
                                                const float* __restrict__ q,
                                                const uint16_t* __restrict__ cache,
                                                size_t seq_stride, int cap,
                                                const int32_t* __restrict__ row_pos,
                                                const int32_t* __restrict__ row_valid,
                                                float scale, float* __restrict__ part,
                                                int32_t* __restrict__ counters,
                                                uint16_t* __restrict__ out) {
  constexpr int KL = DH + 8;            // padded LDS row of K (bf16)
  constexpr int VPT = 64 * DH / 8 / 256;  // uint4 per thread per tile (K or V)
  constexpr int DPL = DH / 64;
  constexpr int RPW = (NR + 3) / 4;     // rows per wave
  __shared__ __align__(16) uint16_t Ks[64 * KL];
  __shared__ __align__(16) uint16_t Vs[64 * DH];
  __shared__ __align__(16) float qs[NR][DH];
  __shared__ __align__(16) float ps[4][64];
  __shared__ int last;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int s = blockIdx.x, h = blockIdx.y;
  const int ngroups = (C + NR - 1) / NR;
  const int b = blockIdx.z / ngroups, g = blockIdx.z % ngroups;
  const int i0 = g * NR, nr = min(NR, C - i0);
  const int D = nh * DH;
  // key limit of every row of the group (block-uniform, for the split
  // range) and of the rows this wave owns (rows wv + 4x)
  int maxpos = -1;
  int lim[RPW];
#pragma unroll
  for (int x = 0; x < RPW; ++x) lim[x] = -1;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    if (i < nr) {
      const int r = b * C + i0 + i;
      const int li = row_valid[r] ? row_pos[r] : -1;
      maxpos = max(maxpos, li);
#pragma unroll
      for (int x = 0; x < RPW; ++x)
        if (i == wv + 4 * x) lim[x] = li;
    }
  }
  // Splits past the group's last key hold no keys: only splits
  // 0..n_live-1 take part (split 0 always, so a group of invalid rows still
  // writes its zero rows).  An empty split's partial (m = -inf, l = 0,
  // o = 0) has zero weight in the merge, so merging the n_live others gives
  // the all-split merge's values bit for bit, with fewer partials to read.
  const int n_live = max(1, min(n_split, (maxpos + spl) / spl));
  if (s >= n_live) return;
  const int k0 = s * spl, k1 = min(k0 + spl, maxpos + 1);
  const uint16_t* Kc = cache + (size_t)b * seq_stride + (size_t)h * cap * DH;
  const uint16_t* Vc = cache + (size_t)b * seq_stride + (size_t)(nh + h) * cap * DH;
  uint4 kreg[VPT], vreg[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) kreg[u] = vreg[u] = make_uint4(0, 0, 0, 0);
  // the query rows are loaded before the first tile, so storing them to
  // LDS does not wait on the tile
  constexpr int QPT = (NR * DH + 255) / 256;
  float qv[QPT];
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = threadIdx.x + 256 * u, i = e / DH, d = e % DH;
    qv[u] = (e < NR * DH && i < nr) ? q[(size_t)(b * C + i0 + i) * D + h * DH + d] : 0.f;
  }
  if (k0 < k1) attn_load_tile<DH, VPT>(Kc, Vc, k0, cap, kreg, vreg);
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = threadIdx.x + 256 * u;
    if (e < NR * DH) qs[e / DH][e % DH] = qv[u];
  }
  float m[RPW], l[RPW], o[RPW][DPL];
#pragma unroll
  for (int x = 0; x < RPW; ++x) {
    m[x] = -INFINITY;
    l[x] = 0.f;
#pragma unroll
    for (int d = 0; d < DPL; ++d) o[x][d] = 0.f;
  }
  for (int t0 = k0; t0 < k1; t0 += 64) {
    __syncthreads();  // previous tile fully consumed
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int c = threadIdx.x + 256 * u;
      const int key = c / (DH / 8), part8 = c % (DH / 8);
      *(uint4*)(Ks + key * KL + part8 * 8) = kreg[u];
      *(uint4*)(Vs + key * DH + part8 * 8) = vreg[u];
    }
    __syncthreads();
    if (t0 + 64 < k1) attn_load_tile<DH, VPT>(Kc, Vc, t0 + 64, cap, kreg, vreg);  // in flight
    const int j = t0 + lane;
#pragma unroll
    for (int x = 0; x < RPW; ++x) {
      const int i = wv + 4 * x;
      if (i >= NR) break;
      // score of key j for row i
      float sc = 0.f;
      const uint16_t* kr = Ks + lane * KL;
#pragma unroll
      for (int c = 0; c < DH / 8; ++c) {
        const uint4 v = *(const uint4*)(kr + c * 8);
        const float4 qa = *(const float4*)&qs[i][c * 8];
        const float4 qb = *(const float4*)&qs[i][c * 8 + 4];
        sc += qa.x * __uint_as_float(v.x << 16) + qa.y * __uint_as_float(v.x & 0xffff0000u) +
              qa.z * __uint_as_float(v.y << 16) + qa.w * __uint_as_float(v.y & 0xffff0000u) +
              qb.x * __uint_as_float(v.z << 16) + qb.y * __uint_as_float(v.z & 0xffff0000u) +
              qb.z * __uint_as_float(v.w << 16) + qb.w * __uint_as_float(v.w & 0xffff0000u);
      }
      const float si = (j <= lim[x]) ? sc * scale : -INFINITY;
      const float mn = fmaxf(m[x], wave_max(si));
      const float p = (mn == -INFINITY) ? 0.f : __expf(si - mn);
      const float corr = (mn == -INFINITY) ? 1.f : __expf(m[x] - mn);
      l[x] = l[x] * corr + wave_sum(p);
#pragma unroll
      for (int d = 0; d < DPL; ++d) o[x][d] *= corr;
      m[x] = mn;
      // P.V over the 64 keys of the tile (p broadcast from LDS; keys past
      // the end of the split have p = 0)
      ps[wv][lane] = p;
      __builtin_amdgcn_wave_barrier();
      lds_wait();
#pragma unroll
      for (int j4 = 0; j4 < 16; ++j4) {
        const float4 p4 = *(const float4*)&ps[wv][4 * j4];
        const float pp[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
        for (int q2 = 0; q2 < 4; ++q2) {
          const int jj = 4 * j4 + q2;
          if (DPL == 2) {
            const uint32_t uu = *(const uint32_t*)(Vs + jj * DH + lane * 2);
            o[x][0] += pp[q2] * __uint_as_float(uu << 16);
            o[x][DPL - 1] += pp[q2] * __uint_as_float(uu & 0xffff0000u);
          } else {
            o[x][0] += pp[q2] * bf2f(Vs[jj * DH + lane]);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  // partial of each owned row
#pragma unroll
  for (int x = 0; x < RPW; ++x) {
    const int i = wv + 4 * x;
    if (i >= nr) break;
    const int r = b * C + i0 + i;
    float* pp = part + (((size_t)r * nh + h) * n_split + s) * (DH + 2);
#pragma unroll
    for (int d = 0; d < DPL; ++d) st_agent(pp + lane * DPL + d, o[x][d]);
    if (lane == 0) {
      st_agent(pp + DH, m[x]);
      st_agent(pp + DH + 1, l[x]);
    }
  }
  vmem_release();
  __syncthreads();
  int32_t* ctr = counters + (size_t)blockIdx.z * nh + h;
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           n_live - 1;
  __syncthreads();
  if (!last) return;
  if (threadIdx.x == 0) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // merge: wave w merges rows w, w+4
#pragma unroll
  for (int x = 0; x < RPW; ++x) {
    const int i = wv + 4 * x;
    if (i >= nr) break;
    const int r = b * C + i0 + i;
    attn_merge_row<DH>(part + ((size_t)r * nh + h) * n_split * (DH + 2), n_live,
                       row_valid[r] != 0, ps[wv], out + (size_t)r * D + h * DH);
  }
}

// sum / max over lanes 0..15 (DPP inside the first 16-lane row), uniform
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<0x111, 0xf>(0.f, v);
  v += dpp_f<0x112, 0xf>(0.f, v);
  v += dpp_f<0x114, 0xf>(0.f, v);
  v += dpp_f<0x118, 0xf>(0.f, v);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 15));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f<0x111, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x112, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x114, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x118, 0xf>(-INFINITY, v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 15));
}

// key limits of a group's four rows, and this wave's query row (row wv:
// lanes 0..15 hold dims 8*lane..8*lane+7; zeros past the group's rows)
__device__ __forceinline__ void attn4_seg_rows(int z, int h, int C, int ngroups, int D,
                                               const float* __restrict__ q,
                                               const int32_t* __restrict__ row_pos,
                                               const int32_t* __restrict__ row_valid,
                                               float4& q0, float4& q1, int (&lim)[4]) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int b = z / ngroups, i0 = (z % ngroups) * 4, nr = min(4, C - i0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = b * C + i0 + i;
    lim[i] = (i < nr && row_valid[r]) ? row_pos[r] : -1;
  }
  q0 = q1 = make_float4(0.f, 0.f, 0.f, 0.f);
  if (wv < nr && lane < 16) {
    const float* p = q + (size_t)(b * C + i0 + wv) * D + h * 128 + 8 * lane;
    q0 = ld_f4(p);
    q1 = ld_f4(p + 4);
  }
}

// this wave's query row as MFMA A-operand pieces: chunk c = lane (8 dims)
// is k-step c/4, lane group c%4; entry 4*group + row of each step
__device__ __forceinline__ void attn4_store_q(uint4 (*qa)[2][16], float4 q0, float4 q1) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane >= 16) return;
  const float x[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint16_t h0 = f2bf(x[2 * e]), h1 = f2bf(x[2 * e + 1]);
    const uint16_t l0 = f2bf(x[2 * e] - bf2f(h0)), l1 = f2bf(x[2 * e + 1] - bf2f(h1));
    hi[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    lo[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  const int s = lane >> 2, e = 4 * (lane & 3) + wv;
  qa[s][0][e] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  qa[s][1][e] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
}

// Split decode attention over groups of four query rows with 128-dim heads
// (every attention call of such a model: a row's arithmetic does not depend
// on how many rows its group or its call has).  Grid, splits, partials and
// merge as k_s_attn.
// Inside a 64-key tile, wave w takes keys 16w..16w+15 for all rows of the
// group, so each K and V element is read from LDS and widened once per
// block: the scores are one 16x16x32 MFMA chain (query rows as the A
// operand, zero rows past the group; the float32 query split into bf16 high
// and low parts, two products per step, so the scores keep ~16 mantissa
// bits of the query against the 8 of a bf16 query), the softmax runs over
// 16-lane rows, and P.V runs on the vector units with the rows' weights
// broadcast from LDS.  Each wave keeps its own (m, l, o) per row for its
// keys; the four wave states are combined through LDS at the end of the
// split, in wave order.  Every update is an explicit fused multiply-add, so
// a row rounds the same way in the one-row and the multi-row code paths.
template <int DH>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_s_attn4(int C, int nh, int n_split, int spl, const float* __restrict__ q,
          const uint16_t* __restrict__ cache, size_t seq_stride, int cap,
          const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_valid,
          float scale, float* __restrict__ part, int32_t* __restrict__ counters,
          uint16_t* __restrict__ out) {
  static_assert(DH == 128, "four k-steps of 32 dims, two dims per lane");
  constexpr int NR = 4;
  constexpr int KL = DH + 8;
  constexpr int VPT = 64 * DH / 8 / 256;
  constexpr int NS = DH / 32;
  __shared__ __align__(16) uint16_t Ks[64 * KL];
  __shared__ __align__(16) uint16_t Vs[64 * DH];
  __shared__ __align__(16) uint4 qa[NS][2][16];
  __shared__ __align__(16) float ps[4][64];
  __shared__ int last;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int s = blockIdx.x, h = blockIdx.y, z = blockIdx.z;
  const int ngroups = (C + NR - 1) / NR;
  const int b = z / ngroups, i0 = (z % ngroups) * NR, nr = min(NR, C - i0);
  const int D = nh * DH;
  float4 q0, q1;
  int lim[4];
  attn4_seg_rows(z, h, C, ngroups, D, q, row_pos, row_valid, q0, q1, lim);
  const int maxpos = max(max(lim[0], lim[1]), max(lim[2], lim[3]));
  // Splits past the group's last key hold no keys: only splits
  // 0..n_live-1 take part (split 0 always, so a group of invalid rows still
  // writes its zero rows).  An empty split's partial (m = -inf, l = 0,
  // o = 0) has zero weight in the merge, so merging the n_live others gives
  // the all-split merge's values bit for bit, with fewer partials to read.
  const int n_live = max(1, min(n_split, (maxpos + spl) / spl));
  if (s >= n_live) return;
  const int k0 = s * spl, k1 = min(k0 + spl, maxpos + 1);
  const uint16_t* Kc = cache + (size_t)b * seq_stride + (size_t)h * cap * DH;
  const uint16_t* Vc = cache + (size_t)b * seq_stride + (size_t)(nh + h) * cap * DH;
  uint4 kreg[VPT], vreg[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) kreg[u] = vreg[u] = make_uint4(0, 0, 0, 0);
  if (k0 < k1) attn_load_tile<DH, VPT>(Kc, Vc, k0, cap, kreg, vreg);
  attn4_store_q(qa, q0, q1);
  float m[4], l[4], o[4][2];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
    o[r][0] = o[r][1] = 0.f;
  }
  const int key16 = lane & 15, grp = lane >> 4;
  for (int t0 = k0; t0 < k1; t0 += 64) {
    __syncthreads();  // previous tile fully consumed, query pieces stored
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int c = threadIdx.x + 256 * u;
      const int key = c / (DH / 8), part8 = c % (DH / 8);
      *(uint4*)(Ks + key * KL + part8 * 8) = kreg[u];
      *(uint4*)(Vs + key * DH + part8 * 8) = vreg[u];
    }
    __syncthreads();
    if (t0 + 64 < k1) attn_load_tile<DH, VPT>(Kc, Vc, t0 + 64, cap, kreg, vreg);  // in flight
    // scores of keys 16wv + key16 for rows 0..3 (lanes 0..15; the other
    // lanes hold the zero rows)
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    const uint16_t* kp = Ks + (16 * wv + key16) * KL + 8 * grp;
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const uint4 kb = *(const uint4*)(kp + 32 * st);
      uint4 ah = make_uint4(0, 0, 0, 0), al = make_uint4(0, 0, 0, 0);
      if (key16 < 4) {
        ah = qa[st][0][4 * grp + key16];
        al = qa[st][1][4 * grp + key16];
      }
      acc = mfma16(ah, kb, acc);
      acc = mfma16(al, kb, acc);
    }
    const int j = t0 + 16 * wv + key16;
    float corr[4] = {1.f, 1.f, 1.f, 1.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (r >= nr) break;
      const float si = (j <= lim[r]) ? acc[r] * scale : -INFINITY;
      const float mn = fmaxf(m[r], row16_max(si));
      const float p = (mn == -INFINITY) ? 0.f : __expf(si - mn);
      corr[r] = (mn == -INFINITY) ? 1.f : __expf(m[r] - mn);
      l[r] = __builtin_fmaf(l[r], corr[r], row16_sum(p));
      m[r] = mn;
      if (lane < 16) ps[wv][4 * lane + r] = p;
    }
    __builtin_amdgcn_wave_barrier();
    lds_wait();
    if (nr == 1) {
      o[0][0] *= corr[0];
      o[0][1] *= corr[0];
#pragma unroll
      for (int kk = 0; kk < 16; ++kk) {
        const float p0 = ps[wv][4 * kk];
        const uint32_t uu = *(const uint32_t*)(Vs + (16 * wv + kk) * DH + lane * 2);
        o[0][0] = __builtin_fmaf(p0, __uint_as_float(uu << 16), o[0][0]);
        o[0][1] = __builtin_fmaf(p0, __uint_as_float(uu & 0xffff0000u), o[0][1]);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        o[r][0] *= corr[r];
        o[r][1] *= corr[r];
      }
#pragma unroll 4
      for (int kk = 0; kk < 16; ++kk) {
        const float4 p4 = *(const float4*)&ps[wv][4 * kk];
        const uint32_t uu = *(const uint32_t*)(Vs + (16 * wv + kk) * DH + lane * 2);
        const float v0 = __uint_as_float(uu << 16), v1 = __uint_as_float(uu & 0xffff0000u);
        o[0][0] = __builtin_fmaf(p4.x, v0, o[0][0]);
        o[0][1] = __builtin_fmaf(p4.x, v1, o[0][1]);
        o[1][0] = __builtin_fmaf(p4.y, v0, o[1][0]);
        o[1][1] = __builtin_fmaf(p4.y, v1, o[1][1]);
        o[2][0] = __builtin_fmaf(p4.z, v0, o[2][0]);
        o[2][1] = __builtin_fmaf(p4.z, v1, o[2][1]);
        o[3][0] = __builtin_fmaf(p4.w, v0, o[3][0]);
        o[3][1] = __builtin_fmaf(p4.w, v1, o[3][1]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // the four waves' states through LDS (over the K tile); row wv combined
  // by wave wv into the split's partial
  float* cb = (float*)Ks;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (r >= nr) break;
    float* e = cb + (wv * 4 + r) * (DH + 2);
    *(float2*)(e + 2 * lane) = make_float2(o[r][0], o[r][1]);
    if (lane == 0) {
      e[DH] = m[r];
      e[DH + 1] = l[r];
    }
  }
  __syncthreads();
  if (wv < nr) {
    float mw[4], lw[4];
    float2 ow[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float* e = cb + (w * 4 + wv) * (DH + 2);
      mw[w] = e[DH];
      lw[w] = e[DH + 1];
      ow[w] = *(const float2*)(e + 2 * lane);
    }
    const float M = fmaxf(fmaxf(mw[0], mw[1]), fmaxf(mw[2], mw[3]));
    float L = 0.f, O0 = 0.f, O1 = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = (mw[w] == -INFINITY) ? 0.f : __expf(mw[w] - M);
      L = __builtin_fmaf(lw[w], f, L);
      O0 = __builtin_fmaf(ow[w].x, f, O0);
      O1 = __builtin_fmaf(ow[w].y, f, O1);
    }
    const int r = b * C + i0 + wv;
    float* pp = part + (((size_t)r * nh + h) * n_split + s) * (DH + 2);
    st_agent(pp + 2 * lane, O0);
    st_agent(pp + 2 * lane + 1, O1);
    if (lane == 0) {
      st_agent(pp + DH, M);
      st_agent(pp + DH + 1, L);
    }
  }
  vmem_release();
  __syncthreads();
  int32_t* ctr = counters + (size_t)z * nh + h;
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           n_live - 1;
  __syncthreads();
  if (!last) return;
  if (threadIdx.x == 0) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (wv < nr) {
    const int r = b * C + i0 + wv;
    attn_merge_row<DH>(part + ((size_t)r * nh + h) * n_split * (DH + 2), n_live,
                       row_valid[r] != 0, ps[wv], out + (size_t)r * D + h * DH);
  }
}

// ---------------------------------------------------------------- router
// One block (16 waves) per 16-row group.  Prologue: y = RMSNorm(h; g)
// into LDS and to xout (bf16, for the experts).  Router logits by MFMA
// (strip x K-quarter per wave), bias, float32 softmax, top-k (larger logit
// first, equal -> lower id), k-th vs (k+1)-th gap; then the grouping of
// (row, slot) pairs by expert (rows ascending) and the list of touched
// experts (ascending id).
template <int MAXT>
__global__ void __launch_bounds__(1024) k_s_router(int R, int H, int E, int topk,
                                                   const float* __restrict__ h,
                                                   const float* __restrict__ g, float eps,
                                                   uint16_t* __restrict__ xout,
                                                   const uint4* __restrict__ Wp,
                                                   const float* __restrict__ bias,
                                                   int32_t* __restrict__ ridx,
                                                   float* __restrict__ rw,
                                                   float* __restrict__ rgap,
                                                   int32_t* __restrict__ ridx_out,
                                                   int32_t* __restrict__ cnt,
                                                   int32_t* __restrict__ off,
                                                   int32_t* __restrict__ ent_row,
                                                   int32_t* __restrict__ ent_slot,
                                                   float* __restrict__ ent_w,
                                                   int32_t* __restrict__ touched,
                                                   int32_t* __restrict__ n_touched) {
  extern __shared__ __align__(16) uint16_t xs[];  // [R][H + XPAD]
  __shared__ f32x4_t red[16 * 64];
  __shared__ float lg[SR_MAX][65];
  __shared__ int sel[SR_MAX * 8];
  __shared__ float selw[SR_MAX * 8];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ldl = H + XPAD, nkt = H / 32;
  const int r0 = blockIdx.x * 16, nloc = min(16, R - r0);
  h += (size_t)r0 * H;
  xout += (size_t)r0 * H;
  ridx += (size_t)r0 * topk;
  rw += (size_t)r0 * topk;
  if (rgap) rgap += r0;
  if (ridx_out) ridx_out += (size_t)r0 * topk;
  // 16 waves = 4 strips x 4 K-quarters; weight tiles first
  const int strip = w >> 2, qk = w & 3, per = nkt / 4;
  const bool live = strip * 16 < E;
  uint4 a[MAXT];
  // (above 10 tiles per wave the prologue runs first: 1024-thread blocks
  // have 128 registers per lane)
  if constexpr (MAXT > 10) norm_rows_lds<MTP_NV(MAXT)>(nloc, H, h, g, eps, xs, ldl);
  preload<MAXT>(Wp + (size_t)(live ? strip : 0) * nkt * 64, qk * per, live ? per : 0, a,
                gridDim.x == 1);
  const float bl = (bias && lane < E) ? bias[lane] : 0.f;
  if constexpr (MAXT <= 10) norm_rows_lds<MTP_NV(MAXT)>(nloc, H, h, g, eps, xs, ldl);
  __syncthreads();
  for (int e = threadIdx.x; e < nloc * H / 8; e += blockDim.x) {
    const int rr = e / (H / 8), c8 = e % (H / 8);
    *(uint4*)(xout + (size_t)rr * H + c8 * 8) = *(const uint4*)(xs + rr * ldl + c8 * 8);
  }
  const int r = lane & 15;
  const uint16_t* xrow = r < nloc ? xs + r * ldl : nullptr;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (live) acc = mma_pre<MAXT, (MAXT % 4 == 0 ? 4 : (MAXT % 5 == 0 ? 5 : MAXT))>(a, qk * per, per, xrow, acc);
  red[w * 64 + lane] = acc;
  __syncthreads();
  if (qk == 0 && live) {
    f32x4_t sacc = red[w * 64 + lane];
    for (int x = 1; x < 4; ++x) sacc += red[(w + x) * 64 + lane];
#pragma unroll
    for (int t = 0; t < 4; ++t) lg[r][strip * 16 + 4 * (lane >> 4) + t] = sacc[t];
  }
  __syncthreads();
  // top-k, one wave per row
  __shared__ __align__(16) float tsc[16][68];
  if (w < nloc) {
    const float lv = lane < E ? lg[w][lane] + bl : -INFINITY;
    lane_topk(lv, E, topk, tsc[w], ridx + (size_t)w * topk, rw + (size_t)w * topk,
              rgap ? rgap + w : nullptr, ridx_out ? ridx_out + (size_t)w * topk : nullptr,
              sel + w * topk, selw + w * topk);
  }
  __syncthreads();
  if (gridDim.x > 1) return;  // several row groups: k_group does the grouping
  // grouping (rows <= 16, each row picks an expert at most once): a row
  // mask per expert (LDS atomics), then one wave derives counts, offsets
  // (prefix sum) and the touched list (ballot); an entry's place within its
  // expert is the number of earlier rows in the expert's mask, so entries
  // are ordered by row.
  __shared__ uint32_t l_mask[64];
  __shared__ int l_off[64];
  const int nent = R * topk;
  if (threadIdx.x < 64) l_mask[threadIdx.x] = 0u;
  __syncthreads();
  if (threadIdx.x < nent) atomicOr(&l_mask[sel[threadIdx.x]], 1u << (threadIdx.x / topk));
  __syncthreads();
  if (w == 0) {
    const int c = lane < E ? __popc(l_mask[lane]) : 0;
    int pre = c;  // inclusive scan over the 64 experts
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(pre, d, MTP_WAVE);
      if (lane >= d) pre += v;
    }
    const int o = pre - c;
    l_off[lane] = o;
    if (lane < E) {
      cnt[lane] = c;
      off[lane] = o;
    }
    const uint64_t has = __ballot(c > 0);
    if (c > 0) touched[__popcll(has & ((1ull << lane) - 1ull))] = lane;
    if (lane == 0) *n_touched = __popcll(has);
  }
  __syncthreads();
  if (threadIdx.x < nent) {
    const int x = threadIdx.x, e = sel[x], r = x / topk;
    const int t = l_off[e] + __popc(l_mask[e] & ((1u << r) - 1u));
    ent_row[t] = r;
    ent_slot[t] = x % topk;
    ent_w[t] = selw[x];
  }
}

// ---------------------------------------------------------------- draft FFN gate/up
// The draft block's FFN gate/up + SwiGLU for up to 16 rows: block = one
// 16-wide intermediate tile (blockIdx.x) of the width-F SwiGLU sgu (gate
// strips, then up strips), K split over 4 waves.  Each wave's first row is
// loaded ahead of the weight tiles and normalised while they are in
// flight; the block then computes RMSNorm(h; g) of its rows into LDS.
// ROLE only names the instance (so profiles separate decode from prefill
// launches; GU_VERIFY / GU_PREFILL name the MoE gate/up of many rows).
enum { GU_VERIFY = 0, GU_DRAFT = 1, GU_PREFILL = 2, GU_DRAFT_PREFILL = 3 };
template <int ROLE, int MAXT>
__global__ void __launch_bounds__(256) k_s_gu(int R, int H, int F, const float* __restrict__ h,
                                              const float* __restrict__ g, float eps,
                                              const uint4* __restrict__ sgu,
                                              uint16_t* __restrict__ act_sh) {
  extern __shared__ __align__(16) uint16_t xs[];
  __shared__ f32x4_t red[2 * 4 * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int it = blockIdx.x, nkt = H / 32, per = nkt / 4, ldl = H + XPAD;
  const uint4* G = sgu + (size_t)it * nkt * 64;
  const uint4* U = sgu + (size_t)(F / 16 + it) * nkt * 64;
  constexpr int NV = MTP_NV(MAXT);
  NormRow<NV> nr0;
  const bool early = w < R;
  if (early) norm_row_load<NV>(H, h + (size_t)w * H, g, nr0);
  uint4 ag_[MAXT], au_[MAXT];
  preload<MAXT>(G, w * per, per, ag_, true);
  preload<MAXT>(U, w * per, per, au_, true);
  const f32x4_t z4 = {0.f, 0.f, 0.f, 0.f};
  f32x4_t cg = z4, cu = z4;
  if (early) norm_row_store<NV>(H, eps, nr0, xs + w * ldl);
  norm_rows_lds<NV>(R, H, h, g, eps, xs, ldl, true);
  __syncthreads();
  // B rows in LDS (lanes past R read a tile row; their columns are not stored)
  mma_pre2<MAXT, (MAXT % 2 == 0 ? MAXT / 2 : MAXT)>(ag_, au_, w * per, per,
                                                     xs + (lane & 15) * ldl, cg, cu);
  cg = block_acc_sum<4>(cg, red);
  cu = block_acc_sum<4>(cu, red + 4 * 64);
  const int t = lane & 15;
  if (w != 0 || t >= R) return;
  const int i = it * 16 + 4 * (lane >> 4);
  uint2 pk;
  pk.x = (uint32_t)f2bf(silu(cg[0]) * cu[0]) | ((uint32_t)f2bf(silu(cg[1]) * cu[1]) << 16);
  pk.y = (uint32_t)f2bf(silu(cg[2]) * cu[2]) | ((uint32_t)f2bf(silu(cg[3]) * cu[3]) << 16);
  *(uint2*)(act_sh + (size_t)t * F + i) = pk;
}

// MoE gate/up for up to 16 rows, persistent streaming form.  Work items:
// (touched routed expert, 16-wide intermediate tile) in touched-list order,
// then the SI/16 tiles of the shared SwiGLU; block b takes items b,
// b + gridDim.x, ...  The R rows are staged in LDS once.  K is split over
// the 4 waves as in k_s_gu; as a wave's product consumes a weight tile, the
// tile's registers are refilled with the block's next item, so the next
// item's loads are in flight during this item's reduction and store (with
// one block per item, blocks that do not fit on the machine at once start
// only when a resident block has finished, after its loads have drained).
// Sums are taken in the same order as k_s_gu's.
template <int MAXT>
__global__ void __launch_bounds__(256) k_s_gu_stream(int R, int H, int I, int SI,
                                                     const uint16_t* __restrict__ xg,
                                                     const uint4* __restrict__ egu,
                                                     size_t e_stride,
                                                     const uint4* __restrict__ sgu,
                                                     const int32_t* __restrict__ cnt,
                                                     const int32_t* __restrict__ off,
                                                     const int32_t* __restrict__ ent_row,
                                                     const int32_t* __restrict__ touched,
                                                     const int32_t* __restrict__ n_touched,
                                                     uint16_t* __restrict__ act,
                                                     uint16_t* __restrict__ act_sh) {
  extern __shared__ __align__(16) uint16_t xs[];  // [R][H + XPAD]
  __shared__ f32x4_t red[2 * 4 * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nkt = H / 32, per = nkt / 4, ldl = H + XPAD, nI = I / 16;
  const int nr = *n_touched * nI, nitems = nr + SI / 16;
  int j = blockIdx.x;
  if (j >= nitems) return;  // block-uniform
  // item -> gate and up strips, expert (-1: shared) and tile
  auto item = [&](int jj, const uint4*& G, const uint4*& U, int& e, int& it) {
    if (jj < nr) {
      e = touched[jj / nI];
      it = jj % nI;
      const uint4* base = egu + (size_t)e * e_stride;
      G = base + (size_t)it * nkt * 64;
      U = base + (size_t)(nI + it) * nkt * 64;
    } else {
      e = -1;
      it = jj - nr;
      G = sgu + (size_t)it * nkt * 64;
      U = sgu + (size_t)(SI / 16 + it) * nkt * 64;
    }
  };
  const uint4 *G, *U;
  int e, it;
  item(j, G, U, e, it);
  // the rows' first 4 KB per wave are loaded before the tiles, so writing
  // them to LDS does not wait on the tiles
  const int nx = R * H / 8;  // 16-byte chunks of the rows
  uint4 xv[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = threadIdx.x + q * 256;
    xv[q] = c < nx ? ((const uint4*)xg)[c] : make_uint4(0, 0, 0, 0);
  }
  uint4 ag_[MAXT], au_[MAXT];
  preload<MAXT>(G, w * per, per, ag_, true);
  preload<MAXT>(U, w * per, per, au_, true);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = threadIdx.x + q * 256;
    if (c < nx) *(uint4*)(xs + (c / (H / 8)) * ldl + (c % (H / 8)) * 8) = xv[q];
  }
  for (int c = threadIdx.x + 1024; c < nx; c += 256)
    *(uint4*)(xs + (c / (H / 8)) * ldl + (c % (H / 8)) * 8) = ((const uint4*)xg)[c];
  __syncthreads();
  const int koff = 8 * (lane >> 4), t = lane & 15;
  for (bool first = true;; first = false) {
    const int jn = j + gridDim.x;
    const bool more = jn < nitems;  // block-uniform
    const uint4 *Gn = G, *Un = U;
    int en = 0, itn = 0;
    if (more) item(jn, Gn, Un, en, itn);
    int n = R, o = 0;
    if (e >= 0) {
      n = cnt[e];
      o = off[e];
    }
    const int row = t < n ? (e >= 0 ? ent_row[o + t] : t) : 0;
    const uint16_t* xrow = xs + row * ldl;
    if (!first) __syncthreads();  // red of the previous item is consumed
    f32x4_t cg = {0.f, 0.f, 0.f, 0.f}, cu = cg;
#pragma unroll
    for (int u = 0; u < MAXT; ++u) {
      if (u < per) {
        const uint4 b = ldx(xrow + (w * per + u) * 32 + koff);
        cg = mfma16(ag_[u], b, cg);
        cu = mfma16(au_[u], b, cu);
        if (more) {
          ag_[u] = ld_tile(Gn + (size_t)(w * per + u) * 64 + lane, true);
          au_[u] = ld_tile(Un + (size_t)(w * per + u) * 64 + lane, true);
        }
      }
    }
    cg = block_acc_sum<4>(cg, red);
    cu = block_acc_sum<4>(cu, red + 4 * 64);
    if (w == 0 && t < n) {
      const int i = it * 16 + 4 * (lane >> 4);
      uint2 pk;
      pk.x = (uint32_t)f2bf(silu(cg[0]) * cu[0]) | ((uint32_t)f2bf(silu(cg[1]) * cu[1]) << 16);
      pk.y = (uint32_t)f2bf(silu(cg[2]) * cu[2]) | ((uint32_t)f2bf(silu(cg[3]) * cu[3]) << 16);
      if (e < 0)
        *(uint2*)(act_sh + (size_t)t * SI + i) = pk;
      else
        *(uint2*)(act + (size_t)(o + t) * I + i) = pk;
    }
    if (!more) break;
    j = jn;
    G = Gn;
    U = Un;
    e = en;
    it = itn;
  }
}

// ---------------------------------------------------------------- MoE down
// MoE down for up to 16 rows: grid (H/16 output strips, NG groups), 4
// waves per block.  The virtual experts -- the touched routed experts in
// ascending id (the router's touched list), then the S shared experts
// (width I each) -- go to wave slot v % (4*NG); a wave streams each of its
// experts' strip tiles in double-buffered batches and accumulates
// w * (Wd[n] . act) per row in LDS.  The contributions
// w * (Wd[n] . act) are summed in 64-bit fixed point (2^-32 units): integer
// addition is exact and associative, so a row's sum does not depend on
// which wave or block handled which expert -- and hence not on the other
// rows of the pass -- and is rounded to float32 once.  Each block stores its
// wave-summed partial (write-through); the last block of the strip adds the
// NG partials and the rounded total to h.  ctr[H/16] must be zero at launch
// (it is left at zero).
// Range: a contribution must be finite and below 2^24 in magnitude; with at
// most 127 contributions per output (E <= 64 routed plus the shared
// experts) the 64-bit sum then stays below 2^63.  Contributions outside
// that range are dropped and set MTP_ERANGE.  Resolution is 2^-32 (finer
// than a float32 ulp for |values| above 2^-9; below that the sum keeps
// an absolute error under 2^-33 per contribution).
constexpr float kFxMax = 16777216.0f;  // 2^24
__device__ __forceinline__ long long fx32(float x, bool& bad) {
  if (!(fabsf(x) < kFxMax)) {
    bad = true;
    return 0;
  }
  return __float2ll_rn(x * 4294967296.0f);
}

template <int NG>
__global__ void __launch_bounds__(256) k_s_down_split(int R, int H, int E, int I, int S,
                                                      const uint16_t* __restrict__ act,
                                                      const uint16_t* __restrict__ act_sh,
                                                      const uint4* __restrict__ edn,
                                                      size_t e_stride,
                                                      const uint4* __restrict__ sdn,
                                                      const int32_t* __restrict__ cnt,
                                                      const int32_t* __restrict__ off,
                                                      const int32_t* __restrict__ ent_row,
                                                      const float* __restrict__ ent_w,
                                                      const int32_t* __restrict__ touched,
                                                      const int32_t* __restrict__ n_touched,
                                                      unsigned long long* __restrict__ part,
                                                      int32_t* __restrict__ ctr,
                                                      float* __restrict__ h,
                                                      int32_t* __restrict__ status) {
  __shared__ long long acc_l[4][SR_MAX][17];
  __shared__ int last;
  const int lane = threadIdx.x & 63;
  // wave-uniform indices: the expert list, counts and offsets are read with
  // scalar loads, so the first weight tiles are issued without waiting on a
  // vector round trip
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nt = blockIdx.x, gq = blockIdx.y;
  const int n_routed = *n_touched, nvirt = n_routed + S;
  for (int e = threadIdx.x; e < 4 * SR_MAX * 17; e += blockDim.x) (&acc_l[0][0][0])[e] = 0;
  __syncthreads();
  const int nkt = I / 32;
  const int t = lane & 15;
  bool bad = false;
  for (int v = gq * 4 + w; v < nvirt; v += NG * 4) {
    const uint4* A;
    const uint16_t* xrow = nullptr;
    int row = -1;
    float wt = 1.f;
    if (v < n_routed) {
      const int e = touched[v];
      const int n = cnt[e], o = off[e];
      A = edn + (size_t)e * e_stride + (size_t)nt * nkt * 64;
      if (t < n) {
        xrow = act + (size_t)(o + t) * I;
        row = ent_row[o + t];
        wt = ent_w[o + t];
      }
    } else {
      const int sx = v - n_routed;
      A = sdn + (size_t)nt * S * nkt * 64 + (size_t)sx * nkt * 64;
      if (t < R) {
        xrow = act_sh + (size_t)t * S * I + (size_t)sx * I;
        row = t;
      }
    }
    const f32x4_t a = sk_range<8>(A, 0, nkt, xrow, f32x4_t{0.f, 0.f, 0.f, 0.f}, true);
    if (row >= 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) acc_l[w][row][4 * (lane >> 4) + q] += fx32(wt * a[q], bad);
    }
  }
  if (bad) set_status(status, MTP_ERANGE);
  __syncthreads();
  const int rr = threadIdx.x >> 4, f = threadIdx.x & 15;
  unsigned long long* pp = part + ((size_t)gq * R + rr) * H + nt * 16 + f;
  if (rr < R)
    __hip_atomic_store(pp,
                       (unsigned long long)(acc_l[0][rr][f] + acc_l[1][rr][f] + acc_l[2][rr][f] +
                                            acc_l[3][rr][f]),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  vmem_release();
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(ctr + nt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           NG - 1;
  __syncthreads();
  if (!last) return;
  if (threadIdx.x == 0) __hip_atomic_store(ctr + nt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (rr < R) {
    long long sum = 0;
#pragma unroll
    for (int x = 0; x < NG; ++x)
      sum += (long long)__hip_atomic_load(part + ((size_t)x * R + rr) * H + nt * 16 + f,
                                          __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    h[(size_t)rr * H + nt * 16 + f] += (float)sum * 2.3283064365386963e-10f;  // 2^-32
  }
}

// ---------------------------------------------------------------- MoE down (slots)
// 17..64 rows (few entries per expert, where a block of 16 output
// features x 16 entries with K split over its 4 waves keeps more blocks in
// flight than the grouped GEMM's 64-entry tiles): block = (16 output
// features, expert y, cpb 16-entry chunks from z*16*cpb).  A routed
// expert's wave tiles (I/128 <= MAXT) are loaded once and applied to the
// block's chunks in turn; the shared block (K = SI) streams its tiles per chunk (the shared
// weights stay in L2), so the registers are sized for one expert's K.
// Routed y < E: slot[(row*(k+1) + slot)][n] = w * (Wd_y[n] . act_t);
// y == E: slot[(r*(k+1) + k)][n] = Wsd[n] . act_sh[r] (the shared experts
// as one width-SI SwiGLU).  k_combine_norm then adds the k+1 slots of
// each row to h in a fixed order.
template <int MAXT>
__global__ void __launch_bounds__(256) k_s_down_slot(int cpb, int R, int E, int topk, int H,
                                                     int I, int SI,
                                                     const uint16_t* __restrict__ act,
                                                     const uint16_t* __restrict__ act_sh,
                                                     const uint4* __restrict__ edn,
                                                     size_t e_stride,
                                                     const uint4* __restrict__ sdn,
                                                     const int32_t* __restrict__ cnt,
                                                     const int32_t* __restrict__ off,
                                                     const int32_t* __restrict__ ent_row,
                                                     const int32_t* __restrict__ ent_slot,
                                                     const float* __restrict__ ent_w,
                                                     float* __restrict__ slot) {
  __shared__ f32x4_t red[4 * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nt = blockIdx.x, e = blockIdx.y, tb = blockIdx.z * 16 * cpb;
  const bool dense = e == E;
  int n = R, o = 0;
  if (!dense) {
    n = cnt[e];
    o = off[e];
  }
  if (tb >= n) return;
  const int K = dense ? SI : I, nkt = K / 32, per = nkt / 4;
  const uint4* A = dense ? sdn + (size_t)nt * nkt * 64
                         : edn + (size_t)e * e_stride + (size_t)nt * nkt * 64;
  // Chunk c's rows: entries tb + 16c + (lane & 15).
  auto chunk_rows = [&](int c, const uint16_t*& xrow, int& row, int& sl, float& wt) {
    const int t = tb + 16 * c + (lane & 15);
    xrow = nullptr;
    row = 0;
    sl = topk;
    wt = 1.f;
    if (t < n) {
      if (dense) {
        xrow = act_sh + (size_t)t * SI;
        row = t;
      } else {
        xrow = act + (size_t)(o + t) * I;
        row = ent_row[o + t];
        sl = ent_slot[o + t];
        wt = ent_w[o + t];
      }
    }
  };
  auto store = [&](int c, f32x4_t acc, int row, int sl, float wt) {
    const int t = tb + 16 * c + (lane & 15);
    if (w == 0 && t < n) {
      float4* dst =
          (float4*)(slot + ((size_t)row * (topk + 1) + sl) * H + nt * 16 + 4 * (lane >> 4));
      *dst = make_float4(wt * acc[0], wt * acc[1], wt * acc[2], wt * acc[3]);
    }
  };
  const f32x4_t z4 = {0.f, 0.f, 0.f, 0.f};
  if (dense) {  // the shared block streams its tiles per chunk (double-buffered)
    for (int c = 0; c < cpb; ++c) {
      if (tb + 16 * c >= n) break;  // block-uniform
      if (c > 0) __syncthreads();
      const uint16_t* xrow;
      int row, sl;
      float wt;
      chunk_rows(c, xrow, row, sl, wt);
      f32x4_t acc = sk_range<4>(A, w * per, (w + 1) * per, xrow, z4, n <= 16 * cpb);
      acc = block_acc_sum<4>(acc, red);
      store(c, acc, row, sl, wt);
    }
    return;
  }
  // a routed expert's wave tiles (I/128 <= MAXT) stay in registers; each
  // chunk's B operands are all loaded before its products
  uint4 a[MAXT];
  preload<MAXT>(A, w * per, per, a, n <= 16 * cpb);  // read by this block only
  for (int c = 0; c < cpb; ++c) {
    if (tb + 16 * c >= n) break;  // block-uniform
    if (c > 0) __syncthreads();
    const uint16_t* xrow;
    int row, sl;
    float wt;
    chunk_rows(c, xrow, row, sl, wt);
    f32x4_t acc = mma_pre<MAXT>(a, w * per, per, xrow, z4);
    acc = block_acc_sum<4>(acc, red);
    store(c, acc, row, sl, wt);
  }
}

// Grouping of (row, slot) pairs by expert for any number of rows: counts,
// offsets (ascending expert id), one entry per pair, and the chunk-block
// prefix cbp of the grouped GEMMs' work items (chunks of 16*cpb entries;
// cbp[E + 1] adds the chunks of the R rows through the shared experts).
// Entries of one expert are placed through LDS atomics, so their order
// inside the expert varies between runs; every value computed from them
// does not (an entry's row and slot travel with it and the MFMA columns
// are independent).
__global__ void __launch_bounds__(1024) k_group(int R, int E, int topk,
                                                const int32_t* __restrict__ ridx,
                                                const float* __restrict__ rw,
                                                int32_t* __restrict__ cnt,
                                                int32_t* __restrict__ off,
                                                int32_t* __restrict__ ent_row,
                                                int32_t* __restrict__ ent_slot,
                                                float* __restrict__ ent_w, int cpb,
                                                int32_t* __restrict__ cbp) {
  __shared__ int l_cnt[64], l_off[64], l_cur[64];
  if (threadIdx.x < 64) {
    l_cnt[threadIdx.x] = 0;
    l_cur[threadIdx.x] = 0;
  }
  __syncthreads();
  const int n = R * topk;
  for (int x = threadIdx.x; x < n; x += blockDim.x) atomicAdd(&l_cnt[ridx[x]], 1);
  __syncthreads();
  if (threadIdx.x < 64) {
    const int e = threadIdx.x;
    int o = 0;
    for (int y = 0; y < e; ++y) o += l_cnt[y];
    l_off[e] = o;
    if (e < E) {
      cnt[e] = l_cnt[e];
      off[e] = o;
    }
    // chunk blocks of 16*cpb entries per expert, prefix over the experts
    const int ch = 16 * cpb, nb = e < E ? (l_cnt[e] + ch - 1) / ch : 0;
    int pre = nb;  // inclusive scan over the 64 lanes
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(pre, d, MTP_WAVE);
      if (e >= d) pre += v;
    }
    if (e < E) cbp[e] = pre - nb;
    if (e == 63) {
      cbp[E] = pre;
      cbp[E + 1] = pre + (R + ch - 1) / ch;
    }
  }
  __syncthreads();
  for (int x = threadIdx.x; x < n; x += blockDim.x) {
    const int e = ridx[x];
    const int t = l_off[e] + atomicAdd(&l_cur[e], 1);
    ent_row[t] = x / topk;
    ent_slot[t] = x % topk;
    ent_w[t] = rw[x];
  }
}

// ---------------------------------------------------------------- LM head
// Block = 4 vocabulary strips (64 rows) x RG 16-row groups (blockIdx.y)
// of the nr input rows X (bf16): each weight tile feeds RG MFMAs.  Per row
// the best logit, its id (lowest on ties) and the second best.
// XL (one row group of more than a few rows): the block's rows are staged
// in LDS once ([16][H + XPAD], dynamic) instead of every wave reading them
// from L2 beside its weight tiles.
// NV > 0 (with XL; NV float4 per lane of a row): the rows are the RMSNorm
// (gain gn) of the float32 rows hx[hidx[o]] (hidx NULL: hx[o]), computed by
// each block while its first weight tiles load -- wave w takes rows w,
// w + 4, ... with k_norm_rows's arithmetic, so the values are its values --
// and block 0 also writes them as float32 to yf[o] (optional); X is unused.
template <int RG, bool XL = false, int NV = 0>
__global__ void __launch_bounds__(256) k_s_lm(int nr, int V, int H, const uint16_t* __restrict__ X,
                                              const uint4* __restrict__ Wp,
                                              float* __restrict__ logits, size_t ldl,
                                              float* __restrict__ pv, int32_t* __restrict__ pi,
                                              float* __restrict__ p2, const float* __restrict__ hx,
                                              const int32_t* __restrict__ hidx,
                                              const float* __restrict__ gn, float eps,
                                              float* __restrict__ yf) {
  constexpr int BT = 4;  // A tiles per batch (each used by RG MFMAs)
  extern __shared__ __align__(16) uint16_t xs[];
  __shared__ float bv[4][16 * RG], sv[4][16 * RG];
  __shared__ int bi[4][16 * RG];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int nkt = H / 32;
  const int nt = blockIdx.x * 4 + wv;
  const int r0 = blockIdx.y * 16 * RG;
  const int r = lane & 15, koff = 8 * (lane >> 4);
  const uint16_t* xrow[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g)
    xrow[g] = r0 + 16 * g + r < nr ? X + (size_t)(r0 + 16 * g + r) * H : nullptr;
  const bool live = nt * 16 < V;
  f32x4_t acc[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g) acc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if constexpr (XL) {
    static_assert(RG == 1, "rows staged for one row group");
    constexpr int XC = 16 * 2048 / 8 / 256;  // 16-byte row chunks per thread (H <= 2048)
    const int ldx_l = H + XPAD, nrow = min(16, nr - r0), nx = nrow * H / 8;
    const uint4* A = Wp + (size_t)nt * nkt * 64;
    uint4 a[8];
    if constexpr (NV > 0) {
      // the first tile batch in flight, then the rows' RMSNorm into LDS
#pragma unroll
      for (int u = 0; u < 8; ++u)
        a[u] = (live && u < nkt) ? ld_tile(A + (size_t)u * 64 + lane, true) : make_uint4(0, 0, 0, 0);
      const int n4 = H / 256;
      for (int q = wv; q < nrow; q += 4) {
        NormRow<NV> nw;
        norm_row_load<NV>(H, hx + (size_t)(hidx ? hidx[r0 + q] : r0 + q) * H, gn, nw);
        float ss = 0.f;
#pragma unroll
        for (int u = 0; u < NV; ++u)
          ss += nw.x[u].x * nw.x[u].x + nw.x[u].y * nw.x[u].y + nw.x[u].z * nw.x[u].z +
                nw.x[u].w * nw.x[u].w;
        ss = wave_sum(ss);
        const float rinv = rsqrtf(ss / (float)H + eps);
#pragma unroll
        for (int u = 0; u < NV; ++u) {
          if (u < n4) {
            const float4 y = make_float4(nw.x[u].x * rinv * nw.g[u].x, nw.x[u].y * rinv * nw.g[u].y,
                                         nw.x[u].z * rinv * nw.g[u].z, nw.x[u].w * rinv * nw.g[u].w);
            const int j4 = u * 64 + lane;
            if (yf && blockIdx.x == 0) ((float4*)(yf + (size_t)(r0 + q) * H))[j4] = y;
            uint2 pk;
            pk.x = (uint32_t)f2bf(y.x) | ((uint32_t)f2bf(y.y) << 16);
            pk.y = (uint32_t)f2bf(y.z) | ((uint32_t)f2bf(y.w) << 16);
            *(uint2*)(xs + q * ldx_l + 4 * j4) = pk;
          }
        }
      }
    } else {
      // row loads first, then the first tile batch: writing the rows to LDS
      // waits on the row loads only
      uint4 xv[XC];
#pragma unroll
      for (int q = 0; q < XC; ++q) {
        const int c = threadIdx.x + 256 * q;
        xv[q] = c < nx ? ((const uint4*)(X + (size_t)r0 * H))[c] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        a[u] = (live && u < nkt) ? ld_tile(A + (size_t)u * 64 + lane, true) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int q = 0; q < XC; ++q) {
        const int c = threadIdx.x + 256 * q;
        if (c < nx) *(uint4*)(xs + (c / (H / 8)) * ldx_l + (c % (H / 8)) * 8) = xv[q];
      }
    }
    __syncthreads();
    if (live) acc[0] = sk_range_lx<8>(A, 0, nkt, xs + (r < nrow ? r : 0) * ldx_l, acc[0], true, a);
  } else if (live) {
    if (RG == 1) {
      acc[0] = sk_range(Wp + (size_t)nt * nkt * 64, 0, nkt, xrow[0], acc[0], true);
    } else {
      const uint4* A = Wp + (size_t)nt * nkt * 64;
      const uint4 z = make_uint4(0, 0, 0, 0);
      for (int t0 = 0; t0 < nkt; t0 += BT) {
        uint4 a[BT], b[RG][BT];
#pragma unroll
        for (int u = 0; u < BT; ++u) a[u] = t0 + u < nkt ? ld_tile(A + (size_t)(t0 + u) * 64 + lane, true) : z;
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
          for (int u = 0; u < BT; ++u)
            b[g][u] = (t0 + u < nkt && xrow[g]) ? ldx(xrow[g] + (t0 + u) * 32 + koff) : z;
#pragma unroll
        for (int u = 0; u < BT; ++u)
#pragma unroll
          for (int g = 0; g < RG; ++g) acc[g] = mfma16(a[u], b[g][u], acc[g]);
      }
    }
  }
  const int v0 = nt * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int g = 0; g < RG; ++g) {
    const int row = r0 + 16 * g + r;
    float b1 = -INFINITY, b2 = -INFINITY;
    int id = 1 << 30;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int v = v0 + t;
      const float x = (live && v < V) ? acc[g][t] : -INFINITY;
      if (logits && row < nr && live && v < V) logits[(size_t)row * ldl + v] = x;
      if (x > b1) {
        b2 = b1;
        b1 = x;
        id = v;
      } else if (x > b2) {
        b2 = x;
      }
    }
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float ob1 = __shfl_xor(b1, o, MTP_WAVE), ob2 = __shfl_xor(b2, o, MTP_WAVE);
      const int oid = __shfl_xor(id, o, MTP_WAVE);
      if (ob1 > b1 || (ob1 == b1 && oid < id)) {
        b2 = fmaxf(b1, ob2);
        b1 = ob1;
        id = oid;
      } else {
        b2 = fmaxf(b2, ob1);
      }
    }
    if (lane < 16) {
      bv[wv][16 * g + lane] = b1;
      sv[wv][16 * g + lane] = b2;
      bi[wv][16 * g + lane] = id;
    }
  }
  __syncthreads();
  if (threadIdx.x < 16 * RG && r0 + (int)threadIdx.x < nr) {
    const int rr = threadIdx.x;
    float c1 = bv[0][rr], c2 = sv[0][rr];
    int cid = bi[0][rr];
    for (int x = 1; x < 4; ++x) {
      const float ob1 = bv[x][rr], ob2 = sv[x][rr];
      const int oid = bi[x][rr];
      if (ob1 > c1 || (ob1 == c1 && oid < cid)) {
        c2 = fmaxf(c1, ob2);
        c1 = ob1;
        cid = oid;
      } else {
        c2 = fmaxf(c2, ob1);
      }
    }
    const size_t o = (size_t)(r0 + rr) * gridDim.x + blockIdx.x;
    pv[o] = c1;
    pi[o] = cid;
    p2[o] = c2;
  }
}

}  // namespace mtp
