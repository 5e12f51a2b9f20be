// Grouped MoE products for passes of more than 16 rows (prefill, large
// verify batches): per expert a GEMM over its entries, tiled so that each
// weight tile feeds 64 entries and each staged row tile feeds 128 output
// features.
//
// Block = 4 waves = 128 output features (wave w: two 16-wide strips,
// features 32w..32w+31 of the block) x 64 entries (four MFMA row tiles).
// The entries' rows are staged through LDS in K chunks of 128 columns,
// double-buffered (the next chunk's global loads fly during the current
// chunk's products); each wave loads its own weight tiles (the packed
// operand tiles of kernels_mfma.h) straight from memory.  Per k-step a
// wave issues 4 (down: 2) weight-tile loads and 4 LDS row reads for 16
// (down: 8) MFMAs.  K is summed in one chain per output tile, in order.
//
// Work items come from the compact grid of k_group (cbp with 64-entry
// chunk blocks): the routed chunk blocks x the N-blocks of one expert, then
// the shared experts' chunk blocks x theirs.
#pragma once
#include "kernels_small.h"

namespace mtp {

constexpr int kGemmM = 64;             // entries per block
constexpr int kGemmN = 128;            // output features per block
constexpr int kGemmKC = 128;           // K columns per LDS stage
constexpr int kGemmLd = kGemmKC + 8;   // LDS row stride (bf16)

// item b: expert e (E = the shared experts), chunk z of 64 entries, N-block
// nb; false past the last item
__device__ __forceinline__ bool gemm_item(int b, int E, int nbr, int nbs,
                                          const int32_t* __restrict__ cbp, int& e, int& z,
                                          int& nb) {
  const int nr = cbp[E] * nbr;
  if (b < nr) {
    nb = b % nbr;
    e = chunk_block_expert(b / nbr, E, cbp, z);
    return true;
  }
  const int bb = b - nr;
  e = E;
  nb = bb % nbs;
  z = bb / nbs;
  return cbp[E] + z < cbp[E + 1];
}

// The 64 rows x 128 columns of one K chunk: thread piece u (of 4) is row
// (tid + 256u) / 16, 8 columns at 8 * ((tid + 256u) % 16).
struct RowStage {
  const uint16_t* src[4];  // the piece's row at column 0 (NULL: a row past the entries)
  uint4 v[4];
  __device__ __forceinline__ void load(int k0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = src[u] ? *(const uint4*)(src[u] + k0) : make_uint4(0, 0, 0, 0);
  }
  __device__ __forceinline__ void store(uint16_t* xs) const {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int p = threadIdx.x + 256 * u;
      *(uint4*)(xs + (p >> 4) * kGemmLd + 8 * (p & 15)) = v[u];
    }
  }
};

// Grouped gate/up + SwiGLU.  Routed expert e: entries off[e].. (rows
// ent_row[]) of xg (normalised bf16 rows [R][H]) -> act[entry][I]; shared
// (e == E): rows 0..R-1 -> act_sh[row][SI] (the shared experts as one
// width-SI SwiGLU).  ROLE only names the instance.
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
  const int s0 = nb * (kGemmN / 16) + 2 * w;  // this wave's first gate strip
  const uint4* Ag = base + (size_t)s0 * nkt * 64 + lane;
  const uint4* Au = base + (size_t)(ns + s0) * nkt * 64 + lane;
  const bool once = n <= kGemmM;  // the expert's tiles are read by this chunk only
  RowStage st;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int t = t0 + ((threadIdx.x + 256 * u) >> 4);
    const int row = t < n ? (dense ? t : ent_row[o + t]) : -1;
    st.src[u] = row >= 0 ? xg + (size_t)row * H + 8 * ((threadIdx.x + 256 * u) & 15) : nullptr;
  }
  st.load(0);
  st.store(xs[0]);
  const f32x4_t z4 = {0.f, 0.f, 0.f, 0.f};
  f32x4_t cg[2][4], cu[2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) cg[j][mt] = cu[j][mt] = z4;
  const int nch = H / kGemmKC;
  for (int kc = 0; kc < nch; ++kc) {
    const int buf = kc & 1;
    uint4 ag[4][2], au[4][2];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const size_t tt = (size_t)j * nkt * 64 + (size_t)(kc * 4 + ks) * 64;
        ag[ks][j] = ld_tile(Ag + tt, once);
        au[ks][j] = ld_tile(Au + tt, once);
      }
    if (kc + 1 < nch) st.load((kc + 1) * kGemmKC);
    __syncthreads();  // chunk kc is in xs[buf]; everyone is done with xs[buf ^ 1]
    const uint16_t* xb = xs[buf] + i16 * kGemmLd + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      uint4 bx[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) bx[mt] = *(const uint4*)(xb + mt * 16 * kGemmLd + 32 * ks);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          cg[j][mt] = mfma16(ag[ks][j], bx[mt], cg[j][mt]);
          cu[j][mt] = mfma16(au[ks][j], bx[mt], cu[j][mt]);
        }
    }
    if (kc + 1 < nch) st.store(xs[buf ^ 1]);
  }
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int t = t0 + mt * 16 + i16;
    if (t >= n) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = (s0 + j) * 16 + 4 * g;
      uint2 pk;
      pk.x = (uint32_t)f2bf(silu(cg[j][mt][0]) * cu[j][mt][0]) |
             ((uint32_t)f2bf(silu(cg[j][mt][1]) * cu[j][mt][1]) << 16);
      pk.y = (uint32_t)f2bf(silu(cg[j][mt][2]) * cu[j][mt][2]) |
             ((uint32_t)f2bf(silu(cg[j][mt][3]) * cu[j][mt][3]) << 16);
      if (dense) *(uint2*)(act_sh + (size_t)t * SI + f) = pk;
      else *(uint2*)(act + (size_t)(o + t) * I + f) = pk;
    }
  }
}

// Grouped MoE down into per-(row, slot) partials: routed expert e,
// entry t: slot[(row * (k+1) + slot)][n] = w * (Wd_e[n] . act[entry]);
// shared (e == E): slot[(r * (k+1) + k)][n] = Wsd[n] . act_sh[r] (K = SI).
// k_combine_norm then adds the k+1 slots of each row to h in a fixed order.
__global__ void __launch_bounds__(256) k_down_gemm(int R, int E, int topk, int H, int I, int SI,
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
  const uint4* A = (dense ? sdn : edn + (size_t)e * e_stride) + (size_t)s0 * nkt * 64 + lane;
  const bool once = n <= kGemmM;
  RowStage st;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int t = t0 + ((threadIdx.x + 256 * u) >> 4);
    const uint16_t* rowp = dense ? act_sh + (size_t)t * SI : act + (size_t)(o + t) * I;
    st.src[u] = t < n ? rowp + 8 * ((threadIdx.x + 256 * u) & 15) : nullptr;
  }
  st.load(0);
  st.store(xs[0]);
  const f32x4_t z4 = {0.f, 0.f, 0.f, 0.f};
  f32x4_t acc[2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[j][mt] = z4;
  const int nch = K / kGemmKC;
  for (int kc = 0; kc < nch; ++kc) {
    const int buf = kc & 1;
    uint4 a[4][2];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        a[ks][j] = ld_tile(A + (size_t)j * nkt * 64 + (size_t)(kc * 4 + ks) * 64, once);
    if (kc + 1 < nch) st.load((kc + 1) * kGemmKC);
    __syncthreads();
    const uint16_t* xb = xs[buf] + i16 * kGemmLd + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      uint4 bx[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) bx[mt] = *(const uint4*)(xb + mt * 16 * kGemmLd + 32 * ks);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[j][mt] = mfma16(a[ks][j], bx[mt], acc[j][mt]);
    }
    if (kc + 1 < nch) st.store(xs[buf ^ 1]);
  }
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
    for (int j = 0; j < 2; ++j)
      *(float4*)(dst + (s0 + j) * 16) =
          make_float4(wt * acc[j][mt][0], wt * acc[j][mt][1], wt * acc[j][mt][2], wt * acc[j][mt][3]);
  }
}

}  // namespace mtp
