// Tiled products for passes of more than 16 rows (prefill, large verify and
// draft batches): the grouped MoE gate/up and down (per expert a GEMM over
// its entries) and the dense projections (QKV with RoPE and the K/V append,
// O / eh / FFN-down with the residual, the draft FFN gate/up), the latter
// with an optional K split over blocks when there are few tiles.
//
// Block = 4 waves = 128 output features (wave w: two 16-wide strips) x 64
// rows (four MFMA row tiles; the core and the dense kernel take the number
// of row tiles MT as a parameter, 4 in every launch: eight row tiles per
// wave leave one wave per SIMD, which measured slower for the LM head).
// The rows are staged through LDS in K chunks of 128 columns,
// double-buffered; each wave loads its own weight tiles (the packed operand
// tiles of kernels_mfma.h) straight from memory into registers, so that
// they fly during the previous chunk's MFMAs: one matrix, two register sets
// (a chunk ahead); two matrices, one set whose k-steps are reloaded with
// the next chunk's as the MFMAs take them.  Per k-step a wave issues 2
// weight-tile loads per matrix and 4 LDS row reads for 8 MFMAs per matrix.
// K is summed in one chain per output tile, in order.
//
// Work items: (weight slab = 128 features of one matrix, 64-row chunk),
// ordered with the chunks of a slab consecutive; blocks are dispatched to
// the 8 XCDs round-robin, so block b takes item xcd_item(b): each XCD takes
// a contiguous run of items, and the chunks that share a weight slab run
// together on one XCD and read it through one L2.
#pragma once
#include "kernels_small.h"

namespace mtp {

constexpr int kGemmM = 64;             // rows (entries) per block
constexpr int kGemmN = 128;            // output features per block
constexpr int kGemmKC = 128;           // K columns per LDS stage
constexpr int kGemmLd = kGemmKC + 8;   // LDS row stride (bf16)
constexpr int kXcd = 8;                // XCDs the blocks are spread over

// Logical item of block b among `total`: XCD x = b mod 8 takes items
// [x*P, (x+1)*P), P = ceil(total / 8), in dispatch order.  Returns total
// for a block past the last item (the grid is 8 * ceil(bound / 8) for a
// bound >= total).
__device__ __forceinline__ int xcd_item(int b, int total) {
  const int P = (total + kXcd - 1) / kXcd, x = b % kXcd, s = b / kXcd;
  return s < P ? min(x * P + s, total) : total;
}

// Grouped item b (cbp: the grouping kernel's prefix of 64-entry chunk
// blocks, cbp[E] the routed total, cbp[E+1] with the shared rows' chunks):
// expert e (E = the shared experts), chunk z, N-block nb; nbr / nbs
// N-blocks per routed / shared slab.  The items of one expert are its nz
// chunks x nbr N-blocks, chunk fastest.  false past the last item.
__device__ __forceinline__ bool gemm_item(int b, int E, int nbr, int nbs,
                                          const int32_t* __restrict__ cbp, int& e, int& z,
                                          int& nb) {
  const int lane = threadIdx.x & 63;
  const int pv = lane < E ? cbp[lane] : 0x7fffffff;
  const int pe = cbp[E], nzs = cbp[E + 1] - pe;
  const int nr = pe * nbr, total = nr + nzs * nbs;
  const int L = xcd_item(b, total);
  if (L >= total) return false;
  if (L < nr) {
    const int c = L / nbr;  // some chunk block of the expert
    e = __popcll(__ballot(pv <= c)) - 1;
    const int c0 = __shfl(pv, e, MTP_WAVE);
    const int c1 = e + 1 < E ? __shfl(pv, e + 1, MTP_WAVE) : pe;
    const int local = L - c0 * nbr, nz = c1 - c0;
    nb = local / nz;
    z = local % nz;
  } else {
    e = E;
    const int local = L - nr;
    nb = local / nzs;
    z = local % nzs;
  }
  return true;
}

// The 16*MT rows x 128 columns of one K chunk: thread piece u (of MT) is
// row (tid + 256u) / 16, 8 columns at 8 * ((tid + 256u) % 16).
template <int MT = 4>
struct RowStage {
  // the piece's row at column 0; a piece past the entries points at a valid
  // row (its products are discarded), so loads carry no per-lane branch
  const uint16_t* src[MT];
  uint4 v[MT];
  __device__ __forceinline__ void load_set(int k0) {
#pragma unroll
    for (int u = 0; u < MT; ++u) v[u] = *(const uint4*)(src[u] + k0);
  }
  __device__ __forceinline__ void store(uint16_t* xs) const {
#pragma unroll
    for (int u = 0; u < MT; ++u) {
      const int p = threadIdx.x + 256 * u;
      *(uint4*)(xs + (p >> 4) * kGemmLd + 8 * (p & 15)) = v[u];
    }
  }
};

// Row piece u of this thread: row of the chunk and column offset
__device__ __forceinline__ int stage_row(int u) { return (threadIdx.x + 256 * u) >> 4; }
__device__ __forceinline__ int stage_col(int u) { return 8 * ((threadIdx.x + 256 * u) & 15); }

// ld_tile with the non-temporal choice fixed at compile time
template <bool NT>
__device__ __forceinline__ uint4 ld_tile_t(const uint4* p) {
  if constexpr (NT) {
    const u32x4_t x = __builtin_nontemporal_load((const u32x4_t*)p);
    return make_uint4(x[0], x[1], x[2], x[3]);
  } else {
    return *p;
  }
}

// The prefetching form of gemm_core (PF): chunk kc + 1's weight tiles are
// loaded during chunk kc's products (two register sets).  Chunk kc + 1's
// rows are requested before its weights, so staging them into LDS after
// chunk kc's products waits for the rows alone (loads complete in order)
// while the weights stay in flight until chunk kc + 1's products.  Every
// st.src is a row (a piece past the entries points at a valid row whose
// products the caller discards), so the row loads carry no per-lane
// branch.  NT: non-temporal weight loads.  Products and their order are
// those of gemm_core.
template <int NA, int MT, bool NT>
__device__ __forceinline__ void gemm_pipe(const uint4* const (&Wt)[NA][2], int nch,
                                          RowStage<MT>& st, uint16_t* xs0, uint16_t* xs1,
                                          f32x4_t (&acc)[NA][2][MT]) {
  const int lane = threadIdx.x & 63, i16 = lane & 15, g = lane >> 4;
  typedef uint4 WSet[NA][4][2];
  WSet w0, w1;
  auto load_w = [&](WSet& wt, int kc) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < 2; ++j) wt[a][ks][j] = ld_tile_t<NT>(Wt[a][j] + (size_t)(kc * 4 + ks) * 64);
  };
  auto mma = [&](const WSet& wt, const uint16_t* xs) {
    const uint16_t* xb = xs + i16 * kGemmLd + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      uint4 bx[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) bx[mt] = *(const uint4*)(xb + mt * 16 * kGemmLd + 32 * ks);
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[a][j][mt] = mfma16(wt[a][ks][j], bx[mt], acc[a][j][mt]);
    }
  };
  // chunk kc: weights wc, rows in LDS stage xc; wn (chunk kc - 1's weights,
  // used) takes chunk kc + 1, whose rows go to xn after the products
  auto step = [&](int kc, const WSet& wc, WSet& wn, const uint16_t* xc, uint16_t* xn) {
    if (kc + 1 < nch) {
      st.load_set((kc + 1) * kGemmKC);
      load_w(wn, kc + 1);
    }
    __syncthreads();  // xc holds chunk kc; every wave is done reading xn
    mma(wc, xc);
    if (kc + 1 < nch) st.store(xn);
  };
  st.load_set(0);
  load_w(w0, 0);
  st.store(xs0);
  for (int kc = 0; kc < nch; kc += 2) {
    step(kc, w0, w1, xs0, xs1);
    if (kc + 1 >= nch) break;
    step(kc + 1, w1, w0, xs1, xs0);
  }
}

// The one-register-set form of gemm_core: as soon as a k-step's MFMAs have
// taken its weight tiles, the same registers are reloaded with that k-step
// of the next chunk, so those loads fly during the rest of this chunk's
// products; the next chunk's rows are requested before them.  Every st.src
// is a row (as gemm_pipe); NT: non-temporal weight loads.
template <int NA, int MT, bool NT>
__device__ __forceinline__ void gemm_roll(const uint4* const (&Wt)[NA][2], int nch,
                                          RowStage<MT>& st, uint16_t* xs0, uint16_t* xs1,
                                          f32x4_t (&acc)[NA][2][MT]) {
  const int lane = threadIdx.x & 63, i16 = lane & 15, g = lane >> 4;
  uint4 wt[NA][4][2];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int j = 0; j < 2; ++j) wt[a][ks][j] = ld_tile_t<NT>(Wt[a][j] + (size_t)ks * 64);
  st.load_set(0);
  st.store(xs0);
  for (int kc = 0; kc < nch; ++kc) {
    const uint16_t* xb = ((kc & 1) ? xs1 : xs0) + i16 * kGemmLd + 8 * g;
    const bool more = kc + 1 < nch;
    if (more) st.load_set((kc + 1) * kGemmKC);
    __syncthreads();  // chunk kc is staged; every wave is done reading the other stage
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      uint4 bx[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) bx[mt] = *(const uint4*)(xb + mt * 16 * kGemmLd + 32 * ks);
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[a][j][mt] = mfma16(wt[a][ks][j], bx[mt], acc[a][j][mt]);
      if (more) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            wt[a][ks][j] = ld_tile_t<NT>(Wt[a][j] + (size_t)((kc + 1) * 4 + ks) * 64);
      }
    }
    if (more) st.store((kc & 1) ? xs0 : xs1);
  }
}

// acc[a][j][mt] = sum over K of matrix a's strip j (tile stream Wt[a][j],
// lane offset included) times row tile mt (of MT) of the staged rows.  K is a
// multiple of kGemmKC; st.src is set; xs0 / xs1 are the two LDS stages.
// Every st.src must point at a row.  PF: gemm_pipe (chunk kc + 1's loads in
// flight during chunk kc's products, two register sets); else gemm_roll
// (one set, each k-step's tiles reloaded with the next chunk's as soon as
// its MFMAs have taken them: with two matrices, two sets would leave one
// wave per SIMD).
template <int NA, bool PF, int MT = 4>
__device__ __forceinline__ void gemm_core(const uint4* const (&Wt)[NA][2], int K, bool once,
                                          RowStage<MT>& st, uint16_t* xs0, uint16_t* xs1,
                                          f32x4_t (&acc)[NA][2][MT]) {
  const int nch = K / kGemmKC;
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[a][j][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if constexpr (PF) {
    if (once) gemm_pipe<NA, MT, true>(Wt, nch, st, xs0, xs1, acc);
    else gemm_pipe<NA, MT, false>(Wt, nch, st, xs0, xs1, acc);
  } else {
    if (once) gemm_roll<NA, MT, true>(Wt, nch, st, xs0, xs1, acc);
    else gemm_roll<NA, MT, false>(Wt, nch, st, xs0, xs1, acc);
  }
}

// Packed bf16 of four floats
__device__ __forceinline__ uint2 pack4(float a, float b, float c, float d) {
  uint2 p;
  p.x = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
  p.y = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
  return p;
}

// Grouped gate/up + SwiGLU: routed expert e: entries off[e].. (rows
// ent_row[]) of xg (normalised bf16 rows [R][H]) -> act[entry][I]; shared
// (e == E): rows 0..R-1 -> act_sh[row][SI] (the shared experts as one
// width-SI SwiGLU).  ROLE only names the instance (decode or prefill).
template <int ROLE>
__global__ void __launch_bounds__(256) k_gu_gemm(int R, int H, int E, int I, int SI,
                                                 const uint16_t* __restrict__ xg,
                                                 const uint4* __restrict__ egu, size_t e_stride,
                                                 const uint4* __restrict__ sgu,
                                                 const int32_t* __restrict__ cnt,
                                                 const int32_t* __restrict__ off,
                                                 const int32_t* __restrict__ ent_row,
                                                 uint16_t* __restrict__ act,
                                                 uint16_t* __restrict__ act_sh,
                                                 const int32_t* __restrict__ cbp) {
  __shared__ __align__(16) uint16_t xs[2][kGemmM * kGemmLd];
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i16 = lane & 15, g = lane >> 4;
  int e, z, nb;
  if (!gemm_item(blockIdx.x, E, I / kGemmN, SI / kGemmN, cbp, e, z, nb)) return;
  const bool dense = e == E;
  const int n = dense ? R : cnt[e], o = dense ? 0 : off[e], t0 = z * kGemmM;
  if (t0 >= n) return;
  const int W = dense ? SI : I, ns = W / 16, nkt = H / 32;
  const uint4* base = dense ? sgu : egu + (size_t)e * e_stride;
  const int s0 = nb * (kGemmN / 16) + 2 * w;  // this wave's first strip
  const uint4* Wt[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    Wt[0][j] = base + (size_t)(s0 + j) * nkt * 64 + lane;       // gate
    Wt[1][j] = base + (size_t)(ns + s0 + j) * nkt * 64 + lane;  // up
  }
  RowStage<4> st;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int t = min(t0 + stage_row(u), n - 1);  // past the entries: a valid row, discarded
    st.src[u] = xg + (size_t)(dense ? t : ent_row[o + t]) * H + stage_col(u);
  }
  f32x4_t acc[2][2][4];
  gemm_core<2, false>(Wt, H, n <= kGemmM, st, xs[0], xs[1], acc);
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int t = t0 + mt * 16 + i16;
    if (t >= n) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = (s0 + j) * 16 + 4 * g;
      const f32x4_t cg = acc[0][j][mt], cu = acc[1][j][mt];
      const uint2 pk = pack4(silu(cg[0]) * cu[0], silu(cg[1]) * cu[1], silu(cg[2]) * cu[2],
                             silu(cg[3]) * cu[3]);
      if (dense) *(uint2*)(act_sh + (size_t)t * SI + f) = pk;
      else *(uint2*)(act + (size_t)(o + t) * I + f) = pk;
    }
  }
}

// Grouped MoE down into per-(row, slot) partials: routed expert e,
// entry t: slot[(row * (k+1) + slot)][n] = w * (Wd_e[n] . act[entry]);
// shared (e == E): slot[(r * (k+1) + k)][n] = Wsd[n] . act_sh[r] (K = SI).
// k_combine_norm then adds the k+1 slots of each row to h in a fixed order.
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_down_gemm(int R, int E, int topk, int H, int I, int SI,
                                                   const uint16_t* __restrict__ act,
                                                   const uint16_t* __restrict__ act_sh,
                                                   const uint4* __restrict__ edn, size_t e_stride,
                                                   const uint4* __restrict__ sdn,
                                                   const int32_t* __restrict__ cnt,
                                                   const int32_t* __restrict__ off,
                                                   const int32_t* __restrict__ ent_row,
                                                   const int32_t* __restrict__ ent_slot,
                                                   const float* __restrict__ ent_w,
                                                   float* __restrict__ slot,
                                                   const int32_t* __restrict__ cbp) {
  __shared__ __align__(16) uint16_t xs[2][kGemmM * kGemmLd];
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i16 = lane & 15, g = lane >> 4;
  int e, z, nb;
  if (!gemm_item(blockIdx.x, E, H / kGemmN, H / kGemmN, cbp, e, z, nb)) return;
  const bool dense = e == E;
  const int n = dense ? R : cnt[e], o = dense ? 0 : off[e], t0 = z * kGemmM;
  if (t0 >= n) return;
  const int K = dense ? SI : I, nkt = K / 32;
  const int s0 = nb * (kGemmN / 16) + 2 * w;  // this wave's first output strip
  const uint4* base = dense ? sdn : edn + (size_t)e * e_stride;
  const uint4* Wt[1][2];
#pragma unroll
  for (int j = 0; j < 2; ++j) Wt[0][j] = base + (size_t)(s0 + j) * nkt * 64 + lane;
  RowStage<4> st;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int t = min(t0 + stage_row(u), n - 1);  // past the entries: a valid row, discarded
    const uint16_t* rowp = dense ? act_sh + (size_t)t * SI : act + (size_t)(o + t) * I;
    st.src[u] = rowp + stage_col(u);
  }
  f32x4_t acc[1][2][4];
  gemm_core<1, true>(Wt, K, n <= kGemmM, st, xs[0], xs[1], acc);
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int t = t0 + mt * 16 + i16;
    if (t >= n) continue;
    int row = t, sl = topk;
    float wt = 1.f;
    if (!dense) {
      row = ent_row[o + t];
      sl = ent_slot[o + t];
      wt = ent_w[o + t];
    }
    float* dst = slot + ((size_t)row * (topk + 1) + sl) * H + 4 * g;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const f32x4_t a = acc[0][j][mt];
      *(float4*)(dst + (s0 + j) * 16) = make_float4(wt * a[0], wt * a[1], wt * a[2], wt * a[3]);
    }
  }
}

// ---------------------------------------------------------------- dense
// Dense products of the normalised rows X (bf16 [R][ldx]) with a packed
// weight matrix, one epilogue per MODE:
//   DG_SET / DG_ADD: Y[r][n] (=|+=) X[r] . W[n]        (Y float32, stride ldy)
//   DG_SWIGLU: act[r][f] = silu(X[r] . G[f]) * (X[r] . U[f]) (bf16 [R][N]; W
//              holds the N gate strips, then the N up strips)
//   DG_QKV:    [q | k | v] = X . Wqkv^T, RoPE (rotate-half) on q and k,
//              q -> q_out (float32 [R][D]), k and v -> the cache at the row
//              position (valid rows); a block's 128 features lie in one of
//              q, k, v, and wave w takes the strips of dims d and d + dh/2
//              of one head, so the rotation pairs are in its registers.
//   DG_ARGMAX: the LM head: logits X[r] . W[v] for v < N (= the vocabulary;
//              the last block's strips past it are masked), optionally
//              stored to logits[r][ldl], and per row and 128-wide block the
//              best logit, its id (lowest on ties) and the second best, at
//              pv/pi/p2[r * ceil(N/128) + block] (as the LM-head kernels
//              of fewer rows, for k_argmax_final).  Never split.
//   DG_ARGMAX_W: DG_ARGMAX with 256 vocabulary rows per block (wave w:
//              strips 4w..4w+3 as two strip pairs through the two-matrix
//              core), partials per 256-wide block.
// With few tiles the K range is split over S blocks per tile (split sk
// takes K chunks [sk*cps, (sk+1)*cps)): each writes its float32 partial
// sums to part[sk][r][col] and k_dense_reduce adds the S partials in order
// and applies the epilogue.  S = 1 applies it directly.
enum { DG_SET = 0, DG_ADD = 1, DG_QKV = 2, DG_SWIGLU = 3, DG_ARGMAX = 4, DG_ARGMAX_W = 5 };
struct DenseOut {
  float* y;            // DG_SET / DG_ADD
  int ldy;
  uint16_t* act;       // DG_SWIGLU
  int C, nh, dh, cap;  // DG_QKV: rows per sequence, heads, head size, cache capacity
  size_t seq_stride;
  const float2* rope;
  const int32_t* row_pos;
  const int32_t* row_valid;
  uint16_t* cache;
  float* q_out;
  float* logits;       // DG_ARGMAX (NULL: not stored)
  size_t ldl;
  float* pv;
  int32_t* pi;
  float* p2;
};

// Partial columns per row: 2N for DG_SWIGLU (gate, then up), else N
template <int MODE>
__host__ __device__ constexpr int dense_cols(int N) { return MODE == DG_SWIGLU ? 2 * N : N; }

// Epilogue of row r at feature f (a multiple of 4): x0 = the sums of
// features f..f+3; x1 = the up sums (DG_SWIGLU) or those of f + dh/2..
// (DG_QKV, f in the first half of a head), else unused.
template <int MODE>
__device__ __forceinline__ void dense_out(const DenseOut& o, int N, int r, int f,
                                          const float (&x0)[4], const float (&x1)[4]) {
  if constexpr (MODE == DG_SET || MODE == DG_ADD) {
    float* y = o.y + (size_t)r * o.ldy + f;
    float4 v = make_float4(x0[0], x0[1], x0[2], x0[3]);
    if (MODE == DG_ADD) {
      const float4 y0 = ld_f4(y);
      v.x += y0.x;
      v.y += y0.y;
      v.z += y0.z;
      v.w += y0.w;
    }
    *(float4*)y = v;
  } else if constexpr (MODE == DG_SWIGLU) {
    *(uint2*)(o.act + (size_t)r * N + f) = pack4(silu(x0[0]) * x1[0], silu(x0[1]) * x1[1],
                                                 silu(x0[2]) * x1[2], silu(x0[3]) * x1[3]);
  } else {
    const int D = o.nh * o.dh, half = o.dh / 2;
    const int sec = f / D, fs = f - sec * D, hh = fs / o.dh, i = fs % o.dh;  // i < dh/2
    const int valid = o.row_valid[r], pos = o.row_pos[r], b = r / o.C;
    if (sec < 2) {
      const float2* cs = o.rope + (size_t)(valid ? pos : 0) * half + i;
      float y0[4], y1[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float2 c = cs[t];
        y0[t] = x0[t] * c.x - x1[t] * c.y;
        y1[t] = x1[t] * c.x + x0[t] * c.y;
      }
      if (sec == 0) {
        float* qr = o.q_out + (size_t)r * D + hh * o.dh + i;
        *(float4*)qr = make_float4(y0[0], y0[1], y0[2], y0[3]);
        *(float4*)(qr + half) = make_float4(y1[0], y1[1], y1[2], y1[3]);
      } else if (valid) {
        uint16_t* kc = o.cache + (size_t)b * o.seq_stride + ((size_t)hh * o.cap + pos) * o.dh + i;
        *(uint2*)kc = pack4(y0[0], y0[1], y0[2], y0[3]);
        *(uint2*)(kc + half) = pack4(y1[0], y1[1], y1[2], y1[3]);
      }
    } else if (valid) {
      uint16_t* vc =
          o.cache + (size_t)b * o.seq_stride + ((size_t)(o.nh + hh) * o.cap + pos) * o.dh + i;
      *(uint2*)vc = pack4(x0[0], x0[1], x0[2], x0[3]);
      *(uint2*)(vc + half) = pack4(x1[0], x1[1], x1[2], x1[3]);
    }
  }
}

__device__ __forceinline__ void to4(const f32x4_t a, float (&x)[4]) {
  x[0] = a[0];
  x[1] = a[1];
  x[2] = a[2];
  x[3] = a[3];
}

// N output features (multiples of 128, except DG_ARGMAX), K (multiple of
// 128); items = the row chunks x N-blocks x S splits, chunk fastest, then
// split.
template <int MODE, int MT = 4>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_dense_gemm(int R, int N, int K,
                                                    const uint16_t* __restrict__ X, int ldx,
                                                    const uint4* __restrict__ Wp, int S,
                                                    float* __restrict__ part, DenseOut o) {
  constexpr bool WIDE = MODE == DG_ARGMAX_W;
  constexpr bool ARGMAX = MODE == DG_ARGMAX || WIDE;
  constexpr int NA = (MODE == DG_SWIGLU || WIDE) ? 2 : 1;
  constexpr int NBLK = WIDE ? 2 * kGemmN : kGemmN;  // output features per block
  constexpr int RM = 16 * MT;  // rows per block
  __shared__ __align__(16) uint16_t xs[2][RM * kGemmLd];
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i16 = lane & 15, g = lane >> 4;
  const int nz = (R + RM - 1) / RM, nbn = (N + NBLK - 1) / NBLK;
  const int L = xcd_item(blockIdx.x, nz * nbn * S);
  if (L >= nz * nbn * S) return;
  const int z = L % nz, sk = (L / nz) % S, nb = L / nz / S;
  const int t0 = z * RM, nkt = K / 32, nch = K / kGemmKC;
  const int cps = (nch + S - 1) / S, kc0 = sk * cps, nkc = min(cps, nch - kc0);
  // this wave's two strips: a rotate-half pair of one head (DG_QKV), else
  // strips 2w, 2w + 1 of the block
  int sa, sb;
  if (MODE == DG_QKV) {
    const int tph = o.dh / 32, ls = (w / tph) * 2 * tph + w % tph;
    sa = nb * (kGemmN / 16) + ls;
    sb = sa + tph;
  } else {
    sa = nb * (NBLK / 16) + (WIDE ? 4 : 2) * w;
    sb = sa + 1;
  }
  // strips past the packed matrix (the last LM-head block) read strip 0;
  // their results are masked
  const int nstr = (N + 15) / 16;
  const uint4* Wt[NA][2];
#pragma unroll
  for (int a = 0; a < NA; ++a) {
    // DG_SWIGLU: matrix a (gate, up) at strip offset a * N/16; wide
    // DG_ARGMAX: strip pair a of the wave (strips sa + 2a, sb + 2a)
    const int ta = WIDE ? sa + 2 * a : sa, tb = WIDE ? sb + 2 * a : sb;  // strips of the matrix
    const int mo = WIDE ? 0 : a * (N / 16);                               // the matrix's first strip
    Wt[a][0] = Wp + ((size_t)((ta < nstr ? ta : 0) + mo) * nkt + kc0 * 4) * 64 + lane;
    Wt[a][1] = Wp + ((size_t)((tb < nstr ? tb : 0) + mo) * nkt + kc0 * 4) * 64 + lane;
  }
  RowStage<MT> st;
#pragma unroll
  for (int u = 0; u < MT; ++u) {
    const int t = min(t0 + stage_row(u), R - 1);  // past the rows: a valid row, discarded
    st.src[u] = X + (size_t)t * ldx + kc0 * kGemmKC + stage_col(u);
  }
  f32x4_t acc[NA][2][MT];
  gemm_core<NA, NA == 1, MT>(Wt, nkc * kGemmKC, nz == 1, st, xs[0], xs[1], acc);
  const int fa = sa * 16 + 4 * g, fb = sb * 16 + 4 * g;
  if constexpr (ARGMAX) {
    // per row: this lane's 8 logits (ascending ids), then the four lanes
    // of the row, then the four waves (through LDS, in wave order)
    __syncthreads();  // every wave is done with the staged rows
    float* bv = (float*)xs[0];
    float* sv = bv + 4 * RM;
    int* bi = (int*)(sv + 4 * RM);
    // a lane's four logits of a strip are consecutive: one 16-byte store
    // where the row stride and the base allow it (measured on a 1,280-row
    // head writing its 662 MB of logits: 4-byte stores cost ~0.16 ms of
    // its 0.83 ms)
    const bool l16 = ((o.ldl & 3) == 0) && ((reinterpret_cast<uintptr_t>(o.logits) & 15) == 0);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int r = t0 + mt * 16 + i16;
      float b1 = -INFINITY, b2 = -INFINITY;
      int id = 1 << 30;
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int v0 = (j ? fb : fa) + 32 * a;
        if (o.logits && r < R) {
          float* dst = o.logits + (size_t)r * o.ldl + v0;
          const f32x4_t y = acc[a][j][mt];
          if (l16 && v0 + 3 < N) {
            *(float4*)dst = make_float4(y[0], y[1], y[2], y[3]);
          } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              if (v0 + t < N) dst[t] = y[t];
          }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int v = v0 + t;  // ascending ids
          const float x = v < N ? acc[a][j][mt][t] : -INFINITY;
          if (x > b1) {
            b2 = b1;
            b1 = x;
            id = v;
          } else if (x > b2) {
            b2 = x;
          }
        }
      }
#pragma unroll
      for (int sh = 16; sh <= 32; sh <<= 1) {
        const float ob1 = __shfl_xor(b1, sh, MTP_WAVE), ob2 = __shfl_xor(b2, sh, MTP_WAVE);
        const int oid = __shfl_xor(id, sh, MTP_WAVE);
        if (ob1 > b1 || (ob1 == b1 && oid < id)) {
          b2 = fmaxf(b1, ob2);
          b1 = ob1;
          id = oid;
        } else {
          b2 = fmaxf(b2, ob1);
        }
      }
      if (lane < 16) {
        bv[w * RM + mt * 16 + lane] = b1;
        sv[w * RM + mt * 16 + lane] = b2;
        bi[w * RM + mt * 16 + lane] = id;
      }
    }
    __syncthreads();
    const int rr = threadIdx.x;
    if (rr < RM && t0 + rr < R) {
      float c1 = bv[rr], c2 = sv[rr];
      int cid = bi[rr];
      for (int x = 1; x < 4; ++x) {
        const float ob1 = bv[x * RM + rr], ob2 = sv[x * RM + rr];
        const int oid = bi[x * RM + rr];
        if (ob1 > c1 || (ob1 == c1 && oid < cid)) {
          c2 = fmaxf(c1, ob2);
          c1 = ob1;
          cid = oid;
        } else {
          c2 = fmaxf(c2, ob1);
        }
      }
      const size_t po = (size_t)(t0 + rr) * nbn + nb;
      o.pv[po] = c1;
      o.pi[po] = cid;
      o.p2[po] = c2;
    }
    return;
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int r = t0 + mt * 16 + i16;
    if (r >= R) continue;
    if (S > 1) {  // float32 partials of this split
      float* pr = part + ((size_t)sk * R + r) * dense_cols<MODE>(N);
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const f32x4_t v = acc[a][j][mt];
          *(float4*)(pr + a * N + (j ? fb : fa)) = make_float4(v[0], v[1], v[2], v[3]);
        }
      continue;
    }
    float x0[4], x1[4];
    if (MODE == DG_QKV) {
      to4(acc[0][0][mt], x0);
      to4(acc[0][1][mt], x1);
      dense_out<MODE>(o, N, r, fa, x0, x1);
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        to4(acc[0][j][mt], x0);
        to4(acc[NA - 1][j][mt], x1);
        dense_out<MODE>(o, N, r, j ? fb : fa, x0, x1);
      }
    }
  }
}

// The S partials of k_dense_gemm summed in split order, then the
// epilogue: one thread per (row, 4 features) -- for DG_QKV per (row, 4
// dims of the first half of a head and their rotate-half partners).
template <int MODE>
__global__ void __launch_bounds__(256) k_dense_reduce(int R, int N, int S,
                                                      const float* __restrict__ part,
                                                      DenseOut o) {
  const int upr = MODE == DG_QKV ? N / 8 : N / 4;  // units per row
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)R * upr) return;
  const int r = (int)(idx / upr), u = (int)(idx % upr);
  int f, f1;  // the x0 and x1 columns
  if (MODE == DG_QKV) {
    const int D = o.nh * o.dh, qg = o.dh / 8;  // 4-dim groups in half a head
    const int sec = u / (D / 8), rem = u % (D / 8);
    f = sec * D + (rem / qg) * o.dh + 4 * (rem % qg);
    f1 = f + o.dh / 2;
  } else {
    f = 4 * u;
    f1 = MODE == DG_SWIGLU ? N + f : f;
  }
  const size_t rs = (size_t)R * dense_cols<MODE>(N);  // floats per split
  const float* p = part + (size_t)r * dense_cols<MODE>(N);
  float x0[4] = {0.f, 0.f, 0.f, 0.f}, x1[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < S; ++s) {
    const float4 a = ld_f4(p + s * rs + f);
    x0[0] += a.x;
    x0[1] += a.y;
    x0[2] += a.z;
    x0[3] += a.w;
    if (MODE == DG_SWIGLU || MODE == DG_QKV) {
      const float4 b = ld_f4(p + s * rs + f1);
      x1[0] += b.x;
      x1[1] += b.y;
      x1[2] += b.z;
      x1[3] += b.w;
    }
  }
  dense_out<MODE>(o, N, r, f, x0, x1);
}

}  // namespace mtp
