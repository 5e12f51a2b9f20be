// bf16 path for gfx950: weights repacked into MFMA operand tiles for
// v_mfma_f32_16x16x32_bf16, the routing decision and the residual
// combine + RMSNorm shared by the contraction kernels (kernels_small.h).
//
// Packed layout of a matrix W[N][K] (K % 128 == 0): tiles (nt, kt) of
// 16 rows x 32 columns, tile order nt-major then kt, 1 KB per tile; lane l
// of a tile holds W[nt*16 + l%16][kt*32 + 8*(l/16) + 0..7] (zero rows past
// N).  A wave loads one tile with one 16-byte load per lane, contiguous
// across the wave -- exactly the A operand of the MFMA.  The B operand is
// a row-major bf16 activation row: lane l reads row (l%16) columns
// kt*32 + 8*(l/16) .. +7.  The MFMA result lane l holds
// D[4*(l/16) + t][l%16]: features 4*(l/16)+t of the strip for row l%16.
#pragma once
#include "common.h"

namespace mtp {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ldx(const uint16_t* p) { return *(const uint4*)p; }

// One lane's 16 bytes of a weight tile.  Tiles a launch reads once are
// loaded non-temporally (measured: a 330 MB stream reaches 6.9 TB/s this
// way against 6.5 TB/s with ordinary loads).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_tile(const uint4* p, bool nt) {
  if (nt) {
    const u32x4_t x = __builtin_nontemporal_load((const u32x4_t*)p);
    return make_uint4(x[0], x[1], x[2], x[3]);
  }
  return *p;
}

inline size_t packed_elems(int N, int K) {  // in uint4 units
  return (size_t)((N + 15) / 16) * (K / 32) * 64;
}

// one thread per (tile, lane): packed[idx] = 8 bf16 of W
__global__ void k_pack(const uint16_t* __restrict__ W, int N, int K, uint4* __restrict__ out) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nkt = K / 32;
  const size_t total = (size_t)((N + 15) / 16) * nkt * 64;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const size_t tile = idx >> 6;
  const int kt = (int)(tile % nkt), nt = (int)(tile / nkt);
  const int n = nt * 16 + (lane & 15), k = kt * 32 + 8 * (lane >> 4);
  out[idx] = n < N ? ldx(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------- top-k helper
// Router decision for one row, one lane per expert (E <= 64): lv = the
// float32 logit (lanes >= E ignored).  Every lane reads all 64 slots from
// LDS (broadcast reads, issued together) and derives its rank --
// #{j : l_j > l_e or (l_j == l_e and j < e)}, i.e. larger logit first, equal
// logits to the lower id; slots >= E hold -inf and never outrank a finite
// logit, so the loop has no per-expert branch.  The float32 softmax
// probability uses the wave max and a wave sum of the exponentials.  Lanes
// of rank < topk write ridx/rw[rank]; gap = l_(k) - l_(k+1) (0 when k == E).
// sc is 68 floats of wave-private, 16-byte aligned LDS.
__device__ __forceinline__ void lane_topk(float lv, int E, int topk, float* sc, int32_t* ridx,
                                          float* rw, float* gap, int32_t* ridx_out, int* sel,
                                          float* selw) {
  const int lane = threadIdx.x & 63;
  const float v = lane < E ? lv : -INFINITY;
  sc[lane] = v;
  __builtin_amdgcn_wave_barrier();
  lds_wait();
  float4 c[16];
#pragma unroll
  for (int j4 = 0; j4 < 16; ++j4) c[j4] = *(const float4*)(sc + 4 * j4);
  int rank = 0;
#pragma unroll
  for (int j4 = 0; j4 < 16; ++j4) {
    const float vv[4] = {c[j4].x, c[j4].y, c[j4].z, c[j4].w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 4 * j4 + q;
      rank += (int)(vv[q] > v) | (int)((vv[q] == v) & (j < lane));
    }
  }
  const float mx = wave_max(v);
  const float ex = lane < E ? __expf(v - mx) : 0.f;
  const float p = ex / wave_sum(ex);
  __builtin_amdgcn_wave_barrier();
  if (lane < E && rank < topk) {
    ridx[rank] = lane;
    rw[rank] = p;
    if (ridx_out) ridx_out[rank] = lane;
    if (sel) {
      sel[rank] = lane;
      selw[rank] = p;
    }
  }
  if (lane < E && rank == topk - 1) sc[64] = v;
  if (lane < E && rank == topk) sc[65] = v;
  __builtin_amdgcn_wave_barrier();
  lds_wait();
  if (lane == 0 && gap) *gap = topk < E ? sc[64] - sc[65] : 0.f;
}

// h[r] += slot[r][k] (dense) + sum_{j<k} slot[r][j]; then RMSNorm of the
// new h with gain g -> xin (bf16, product input) and/or yf (float32).
// One block of H/4 threads per row, thread j owning columns 4j..4j+3: the
// row, its k+1 slots and the gain are all loaded before any sum (k <= 8).
// slot may be NULL (no MoE contribution to add).
__global__ void __launch_bounds__(512) k_combine_norm(int H, int topk,
                                                      const float* __restrict__ slot,
                                                      float* __restrict__ h,
                                                      const float* __restrict__ g, float eps,
                                                      float* __restrict__ yf,
                                                      uint16_t* __restrict__ xin) {
  __shared__ float red[16];
  const int r = blockIdx.x, j4 = threadIdx.x;
  float4* hr = (float4*)(h + (size_t)r * H);
  float4 v = ld_f4(h + (size_t)r * H + j4 * 4);
  const float4 gv = ld_f4(g + j4 * 4);
  if (slot) {
    const float* s0 = slot + (size_t)r * (topk + 1) * H;
    float4 sv[9];
#pragma unroll
    for (int x = 0; x < 9; ++x)
      sv[x] = x <= topk ? ld_f4(s0 + (size_t)x * H + j4 * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 add = sv[0];
#pragma unroll
    for (int x = 0; x < 9; ++x)
      if (x == topk) add = sv[x];  // the dense (shared) slot first
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      if (x < topk) {
        add.x += sv[x].x;
        add.y += sv[x].y;
        add.z += sv[x].z;
        add.w += sv[x].w;
      }
    }
    v.x += add.x;
    v.y += add.y;
    v.z += add.z;
    v.w += add.w;
    hr[j4] = v;
  }
  float ss = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  ss = block_sum(ss, red);
  const float rinv = rsqrtf(ss / (float)H + eps);
  const float4 y = make_float4(v.x * rinv * gv.x, v.y * rinv * gv.y, v.z * rinv * gv.z,
                               v.w * rinv * gv.w);
  if (yf) ((float4*)(yf + (size_t)r * H))[j4] = y;
  if (xin) {
    uint2 pk;
    pk.x = (uint32_t)f2bf(y.x) | ((uint32_t)f2bf(y.y) << 16);
    pk.y = (uint32_t)f2bf(y.z) | ((uint32_t)f2bf(y.w) << 16);
    ((uint2*)(xin + (size_t)r * H))[j4] = pk;
  }
}

}  // namespace mtp
