// Flash-style causal attention for prefill passes (many query rows of a
// sequence against its cache), 128-dim heads.  Both products on MFMA
// (16x16x32 bf16): the scores S = K Q^T with the float32 query split into
// bf16 high and low parts (two products per k-step, as the decode kernel
// does: the scores keep ~16 mantissa bits of the query), the values
// O^T = V^T P^T with the float32 probabilities split the same way (so the
// weighted sum keeps ~16 bits of each weight before its float32
// accumulation).  Online softmax in float32 per row.
#pragma once
#include "kernels_small.h"

namespace mtp {

// two bf16 parts (high, low) of 8 floats, packed as MFMA operands
__device__ __forceinline__ void split8(const float (&x)[8], uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint16_t h0 = f2bf(x[2 * e]), h1 = f2bf(x[2 * e + 1]);
    const uint16_t l0 = f2bf(x[2 * e] - bf2f(h0)), l1 = f2bf(x[2 * e + 1] - bf2f(h1));
    h[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// Block = 4 waves = 64 query rows (wave w: rows 16w..16w+15 of tile
// blockIdx.x % ntile) of head blockIdx.y of sequence blockIdx.z; the C rows
// of each sequence sit at row_pos[b*C + i] (invalid rows: zeros).  Keys run
// in 64-key tiles up to the largest position of the block's valid rows;
// each row masks keys past its own position.
// SPLIT: the keys are cut into chunks of CH tiles, chunk c = blockIdx.x /
// ntile (a row tile's chunks run in parallel instead of one after the
// other); the block writes each row's unnormalised partial (o, m, l) of its
// chunk to part[((row * nh + head) * n_part + c) * (DH + 2)] -- the split
// partials of the decode attention -- and k_attn_merge combines a row's
// chunks.  A chunk past the tile's last key writes nothing (no row of the
// tile reads it).
//
// Layouts (lane l, g = l/16, i = l%16):
//   S tile q (keys 16q..16q+15 of the key tile): A = K rows (lane: key i,
//     dims 8g.. of the k-step, from the K tile in LDS), B = Q (lane: row i,
//     same dims) -> lane holds S[key 16q + 4g + t][row i], t = 0..3;
//   PV over 32 keys c (S tiles 2c, 2c+1): the contraction order pairs the
//     lane's own scores with the keys it holds, position 8g + j ->
//     key 32c + 4g + j (j < 4) or 32c + 16 + 4g + j - 4 (j >= 4), so
//     B = P needs no data movement and A = V^T reads two 8-byte runs of the
//     V tile, stored transposed in LDS ([dim][key]); the result lane holds
//     O[row i][dim 16d + 4g + t] for dim tile d.
template <int DH, bool SPLIT = false>
__global__ void __launch_bounds__(256) k_flash_prefill(int C, int nh,
                                                       const float* __restrict__ q,
                                                       const uint16_t* __restrict__ cache,
                                                       size_t seq_stride, int cap,
                                                       const int32_t* __restrict__ row_pos,
                                                       const int32_t* __restrict__ row_valid,
                                                       float scale, uint16_t* __restrict__ out,
                                                       int ntile = 0, int CH = 0, int n_part = 0,
                                                       float* __restrict__ part = nullptr) {
  static_assert(DH == 128, "four k-steps of 32 dims");
  constexpr int NS = DH / 32, ND = DH / 16, VL = 64 + 8, KL = DH + 8;
  __shared__ __align__(16) uint16_t vt[DH * VL];  // V tile transposed: [dim][key]
  // K tile as stored ([key][dim]); rows 272 bytes apart, so the 16 lanes of
  // one 16-byte column piece read 16 different bank groups
  __shared__ __align__(16) uint16_t kt[64 * KL];
  __shared__ int s_kmax;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int i16 = lane & 15, g = lane >> 4;
  const int h = blockIdx.y, b = blockIdx.z, D = nh * DH;
  const int tile = SPLIT ? blockIdx.x % ntile : blockIdx.x;
  const int chunk = SPLIT ? blockIdx.x / ntile : 0;
  const int r = tile * 64 + 16 * w + i16;  // this lane's query row (of the sequence)
  const bool rv = r < C && row_valid[(size_t)b * C + r];
  const int rp = rv ? row_pos[(size_t)b * C + r] : -1;
  if (threadIdx.x == 0) s_kmax = 0;
  __syncthreads();
  if (rv) atomicMax(&s_kmax, rp + 1);
  // query operands (high / low parts) of the four k-steps
  uint4 qh[NS], ql[NS];
  {
    const float* qp = q + ((size_t)b * C + (r < C ? r : 0)) * D + (size_t)h * DH + 8 * g;
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      float x[8];
      const float4 a = rv ? ld_f4(qp + 32 * ks) : make_float4(0.f, 0.f, 0.f, 0.f);
      const float4 c = rv ? ld_f4(qp + 32 * ks + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
      split8(x, qh[ks], ql[ks]);
    }
  }
  __syncthreads();
  const int kend = s_kmax < cap ? s_kmax : cap;
  const int kbeg = SPLIT ? chunk * CH * 64 : 0;
  const int kmax = SPLIT ? min(kend, kbeg + CH * 64) : kend;
  if (kbeg >= kmax && SPLIT) return;  // block-uniform
  const uint16_t* Kc = cache + (size_t)b * seq_stride + (size_t)h * cap * DH;
  const uint16_t* Vc = cache + (size_t)b * seq_stride + (size_t)(nh + h) * cap * DH;
  float m = -INFINITY, lsum = 0.f;
  f32x4_t o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d) o[d] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // tiles in flight: this thread's share of the K and V tiles (16-byte
  // pieces).  K: sixteen consecutive lanes read one key's row, so a wave
  // reads four whole rows; the tile is stored in LDS once per block and
  // every wave takes its operands from there (each wave reading its own copy
  // from memory moved four times the bytes; measured on the 1,668-row
  // prefill: 5.28 -> 5.07 ms).
  // V: a thread holds 8 dims of 4 consecutive keys and stores each dim's 4
  // keys as one 8-byte run of the transposed tile (4 LDS stores a tile
  // instead of 32 two-byte ones: 1,668-row prefill 5.08 -> 5.03 ms).
  // Keys past the capacity clamp to its last row and are masked below.  The
  // next tile's loads are issued as soon as the current tile is in LDS, so
  // they fly during its scores, softmax and P.V.
  constexpr int VP = 64 * DH / 8 / 256;
  u32x4_t kr[VP];  // (a native vector: a uint4 array copied to LDS whole went to scratch)
  uint4 vr[VP];
  auto load_k = [&](int k0) {
#pragma unroll
    for (int u = 0; u < VP; ++u) {
      const int c = threadIdx.x + 256 * u;
      const int key = min(k0 + (c >> 4), cap - 1);
      kr[u] = *(const u32x4_t*)(Kc + (size_t)key * DH + (c & 15) * 8);
    }
  };
  static_assert(VP == 4, "a thread holds 8 dims of 4 keys of the V tile");
  const int vq = threadIdx.x & 15, vd = threadIdx.x >> 4;  // keys 4vq.., dims 8vd..
  auto load_v = [&](int k0) {
#pragma unroll
    for (int u = 0; u < VP; ++u) {
      const int key = min(k0 + 4 * vq + u, cap - 1);
      vr[u] = *(const uint4*)(Vc + (size_t)key * DH + vd * 8);
    }
  };
  if (kmax > kbeg) {
    load_k(kbeg);
    load_v(kbeg);
  }
  for (int k0 = kbeg; k0 < kmax; k0 += 64) {
    const bool more = k0 + 64 < kmax;
    __syncthreads();  // the previous tile's scores and P.V are done with the K and V tiles
#pragma unroll
    for (int u = 0; u < VP; ++u) {  // K tile into LDS
      const int c = threadIdx.x + 256 * u;
      *(u32x4_t*)(kt + (c >> 4) * KL + (c & 15) * 8) = kr[u];
    }
    {  // V tile into LDS, transposed: per dim, the thread's four keys as one 8-byte run
      const uint32_t v0[4] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w};
      const uint32_t v1[4] = {vr[1].x, vr[1].y, vr[1].z, vr[1].w};
      const uint32_t v2[4] = {vr[2].x, vr[2].y, vr[2].z, vr[2].w};
      const uint32_t v3[4] = {vr[3].x, vr[3].y, vr[3].z, vr[3].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint16_t* dst = vt + (vd * 8 + 2 * e) * VL + 4 * vq;
        *(uint2*)dst = make_uint2((v0[e] & 0xffffu) | (v1[e] << 16), (v2[e] & 0xffffu) | (v3[e] << 16));
        *(uint2*)(dst + VL) =
            make_uint2((v0[e] >> 16) | (v1[e] & 0xffff0000u), (v2[e] >> 16) | (v3[e] & 0xffff0000u));
      }
    }
    if (more) {
      load_k(k0 + 64);
      load_v(k0 + 64);
    }
    __syncthreads();  // the K and V tiles are in LDS
    // scores, scaled and masked
    float s[4][4];
    float mx = m;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
      const uint16_t* kp0 = kt + (16 * qq + i16) * KL + 8 * g;
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        const uint4 ka = *(const uint4*)(kp0 + 32 * ks);
        acc = mfma16(ka, qh[ks], acc);
        acc = mfma16(ka, ql[ks], acc);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int kp = k0 + 16 * qq + 4 * g + t;
        s[qq][t] = (kp <= rp) ? acc[t] * scale : -INFINITY;
        mx = fmaxf(mx, s[qq][t]);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, MTP_WAVE));
    mx = fmaxf(mx, __shfl_xor(mx, 32, MTP_WAVE));
    const float corr = (mx == -INFINITY) ? 1.f : __expf(m - mx);
    float ps = 0.f;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float p = (mx == -INFINITY) ? 0.f : __expf(s[qq][t] - mx);
        s[qq][t] = p;
        ps += p;
      }
    lsum = __builtin_fmaf(lsum, corr, ps);
    m = mx;
#pragma unroll
    for (int d = 0; d < ND; ++d) o[d] *= corr;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float x[8];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        x[t] = s[2 * c][t];
        x[4 + t] = s[2 * c + 1][t];
      }
      uint4 ph, pl;
      split8(x, ph, pl);
#pragma unroll
      for (int d = 0; d < ND; ++d) {
        const uint16_t* vp = vt + (16 * d + i16) * VL + 32 * c + 4 * g;
        const uint2 a0 = *(const uint2*)vp;
        const uint2 a1 = *(const uint2*)(vp + 16);
        const uint4 av = make_uint4(a0.x, a0.y, a1.x, a1.y);
        o[d] = mfma16(av, ph, o[d]);
        o[d] = mfma16(av, pl, o[d]);
      }
    }
  }
  // the row's sum over its four lanes, then O / l as bf16
  float lt = lsum + __shfl_xor(lsum, 16, MTP_WAVE);
  lt += __shfl_xor(lt, 32, MTP_WAVE);
  if (SPLIT) {
    if (r < C) {
      float* pp = part + ((((size_t)b * C + r) * nh + h) * n_part + chunk) * (DH + 2);
#pragma unroll
      for (int d = 0; d < ND; ++d)
        *(float4*)(pp + 16 * d + 4 * g) = make_float4(o[d][0], o[d][1], o[d][2], o[d][3]);
      if (g == 0) {
        pp[DH] = m;
        pp[DH + 1] = lt;
      }
    }
    return;
  }
  if (r < C) {
    uint16_t* op = out + ((size_t)b * C + r) * D + (size_t)h * DH + 4 * g;
    const float inv = (rv && lt > 0.f) ? 1.f / lt : 0.f;
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      uint2 pk;
      pk.x = (uint32_t)f2bf(o[d][0] * inv) | ((uint32_t)f2bf(o[d][1] * inv) << 16);
      pk.y = (uint32_t)f2bf(o[d][2] * inv) | ((uint32_t)f2bf(o[d][3] * inv) << 16);
      *(uint2*)(op + 16 * d) = pk;
    }
  }
}

// Combines the key chunks of the split prefill attention: one wave per
// (row, head), the row's chunks being those that reach its position
// (ceil(ceil((pos + 1) / 64) / CH)); writes the bf16 row (zeros for an
// invalid row).
template <int DH>
__global__ void __launch_bounds__(256) k_attn_merge(int R, int nh, int CH, int n_part,
                                                    const float* __restrict__ part,
                                                    const int32_t* __restrict__ row_pos,
                                                    const int32_t* __restrict__ row_valid,
                                                    uint16_t* __restrict__ out) {
  __shared__ float ws[4][64];
  const int w = threadIdx.x >> 6, x = blockIdx.x * 4 + w;
  if (x >= R * nh) return;
  const int r = x / nh, h = x % nh;
  const bool valid = row_valid[r] != 0;
  const int n = valid ? min(n_part, ((row_pos[r] + 64) / 64 + CH - 1) / CH) : 0;
  attn_merge_row<DH>(part + ((size_t)r * nh + h) * n_part * (DH + 2), n, valid, ws[w],
                     out + (size_t)r * nh * DH + h * DH);
}

}  // namespace mtp
