// Shared device helpers of the MI355X FastMTP library (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mtp.h"

#define MTP_WAVE 64

namespace mtp {

// ---------------------------------------------------------------- storage
// bf16 is carried as its bit pattern (uint16_t); conversions are exact
// widening and round-to-nearest-even narrowing.
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <bool BF>
struct St;
template <>
struct St<true> {
  using T = uint16_t;
  static __device__ __forceinline__ float ld(const T* p, size_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void st(T* p, size_t i, float v) { p[i] = f2bf(v); }
  // value rounded to the storage type, returned widened
  static __device__ __forceinline__ float rnd(float v) { return bf2f(f2bf(v)); }
};
template <>
struct St<false> {
  using T = float;
  static __device__ __forceinline__ float ld(const T* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void st(T* p, size_t i, float v) { p[i] = v; }
  static __device__ __forceinline__ float rnd(float v) { return v; }
};

// ---------------------------------------------------------------- reductions
// Wave64 reductions with DPP moves (row_shr 1/2/4/8 inside each 16-lane
// row, then row_bcast15 / row_bcast31 across rows; lane 63 ends with the
// total, which readlane broadcasts).  Lanes whose DPP source is outside the
// row keep the identity passed as `old`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float identity, float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(v),
                                                    CTRL, ROW_MASK, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0x111, 0xf>(0.f, v);  // row_shr:1
  v += dpp_f<0x112, 0xf>(0.f, v);  // row_shr:2
  v += dpp_f<0x114, 0xf>(0.f, v);  // row_shr:4
  v += dpp_f<0x118, 0xf>(0.f, v);  // row_shr:8
  v += dpp_f<0x142, 0xa>(0.f, v);  // row_bcast:15
  v += dpp_f<0x143, 0xc>(0.f, v);  // row_bcast:31
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0x111, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x112, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x114, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x118, 0xf>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x142, 0xa>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x143, 0xc>(-INFINITY, v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
// block-wide sum over blockDim.x threads (multiple of 64, <= 1024)
__device__ __forceinline__ float block_sum(float v, float* red /* >= 16 floats */) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}

// 16-byte load of 4 floats through the native vector type: HIP's float4 is
// a struct, and a struct load under a condition can be split into four
// 4-byte loads (four load instructions where one suffices).
__device__ __forceinline__ float4 ld_f4(const float* p) {
  typedef float v4f __attribute__((ext_vector_type(4)));
  const v4f v = *(const v4f*)p;
  return make_float4(v[0], v[1], v[2], v[3]);
}

// Greedy-argmax reduction step: (best value, lowest id on ties, second
// best value) of two partial results.
__device__ __forceinline__ void argmax_combine(float& bv, float& sv, int& bi, float v, float s,
                                               int i) {
  if (v > bv || (v == bv && i < bi)) {
    sv = fmaxf(bv, s);
    bv = v;
    bi = i;
  } else {
    sv = fmaxf(sv, v);
  }
}

// Argmax of row r over its nblk LM-head partials (pv/pi/p2 at
// r*nblk + j) by a 256-thread block: each thread loads its up to 8
// partials per round before combining them (all loads in flight), then a
// wave and a block reduction.  The token is returned (and the best and
// second best values stored) in thread 0.
__device__ __forceinline__ int argmax_row(int r, int nblk, const float* __restrict__ pv,
                                          const int32_t* __restrict__ pi,
                                          const float* __restrict__ p2, float* best = nullptr,
                                          float* second = nullptr) {
  __shared__ float wb[4], ws2[4];
  __shared__ int wi[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float bv = -INFINITY, sv = -INFINITY;
  int bi = 1 << 30;
  for (int j0 = 0; j0 < nblk; j0 += 256 * 8) {
    float v[8], s[8];
    int id[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u * 256 + threadIdx.x;
      const size_t o = (size_t)r * nblk + j;
      const bool ok = j < nblk;
      v[u] = ok ? pv[o] : -INFINITY;
      s[u] = ok ? p2[o] : -INFINITY;
      id[u] = ok ? pi[o] : (1 << 30);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) argmax_combine(bv, sv, bi, v[u], s[u], id[u]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, MTP_WAVE), os = __shfl_xor(sv, o, MTP_WAVE);
    const int oi = __shfl_xor(bi, o, MTP_WAVE);
    argmax_combine(bv, sv, bi, ov, os, oi);
  }
  if (lane == 0) {
    wb[w] = bv;
    ws2[w] = sv;
    wi[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int x = 1; x < 4; ++x) argmax_combine(bv, sv, bi, wb[x], ws2[x], wi[x]);
    if (best) *best = bv;
    if (second) *second = sv;
  }
  return bi;
}

// Wait for this wave's outstanding LDS operations only (lgkmcnt(0); vmcnt
// and expcnt at their maxima, so global loads in flight keep flying).
// Used with a wave barrier when a wave reads back LDS it has just written.
__device__ __forceinline__ void lds_wait() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Cross-workgroup publication without cache maintenance.  The L2 of one
// XCD is not coherent with the others, and a device-scope fence
// (__threadfence) writes back and invalidates the whole L2.  Data that one
// workgroup hands to another inside a kernel is therefore stored and
// loaded with agent-scope atomic accesses (write-through stores and loads
// that do not hit stale L2 lines); vmem_release() orders those stores
// before a following flag atomic by waiting for their completion.
//
// The hand-off (a partial-result merge by the last block of a group):
//   writer: st_agent partials; vmem_release (vmcnt(0): the write-through
//           stores have completed); agent-scope fetch_add on the count.
//   reader: the block whose fetch_add returned the last count waits for
//           that return (vmcnt), passes a workgroup barrier, and only then
//           issues its ld_agent loads -- agent-scope atomic loads, which
//           read at the coherence point and so see every completed store.
// An agent-scope acquire fence (buffer_inv sc1 on gfx950) is what makes
// later *non-atomic* loads observe such stores; every cross-block read here
// is an agent-scope atomic load issued after the count was observed, so
// none is used -- in the last block it costs 1.2-1.5 us per launch of the
// attention and MoE-down kernels (measured), on the step's critical path.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void vmem_release() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
}


// sticky status: the first error code wins
__device__ __forceinline__ void set_status(int32_t* status, int32_t code) {
  atomicCAS(status, 0, code);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

}  // namespace mtp
