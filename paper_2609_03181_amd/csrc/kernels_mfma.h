// bf16 fast path for gfx950: weights repacked into MFMA operand tiles,
// v_mfma_f32_16x16x32_bf16 contractions with fused epilogues, grouped MoE,
// KV-sharing split-K decode attention, LM head with fused argmax.
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

// acc[rt] += strip(16 x K) . X rows, K = nkt*32 (nkt % 4 == 0).  xr[rt] is
// this lane's activation row for r-tile rt, or nullptr (zero column).
template <int RT>
__device__ __forceinline__ void strip_mma(const uint4* __restrict__ A, int nkt,
                                          const uint16_t* const (&xr)[RT], f32x4_t (&acc)[RT]) {
  const int lane = threadIdx.x & 63;
  const int koff = 8 * (lane >> 4);
  const uint4 z = make_uint4(0, 0, 0, 0);
  for (int kt = 0; kt < nkt; kt += 4) {
    uint4 a[4], b[4][RT];
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = A[(size_t)(kt + u) * 64 + lane];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) b[u][rt] = xr[rt] ? ldx(xr[rt] + (kt + u) * 32 + koff) : z;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma16(a[u], b[u][rt], acc[rt]);
  }
}

// two strips sharing the same activation rows (gate and up)
template <int RT>
__device__ __forceinline__ void strip2_mma(const uint4* __restrict__ A0,
                                           const uint4* __restrict__ A1, int nkt,
                                           const uint16_t* const (&xr)[RT], f32x4_t (&acc0)[RT],
                                           f32x4_t (&acc1)[RT]) {
  const int lane = threadIdx.x & 63;
  const int koff = 8 * (lane >> 4);
  const uint4 z = make_uint4(0, 0, 0, 0);
  for (int kt = 0; kt < nkt; kt += 4) {
    uint4 a0[4], a1[4], b[4][RT];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a0[u] = A0[(size_t)(kt + u) * 64 + lane];
      a1[u] = A1[(size_t)(kt + u) * 64 + lane];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) b[u][rt] = xr[rt] ? ldx(xr[rt] + (kt + u) * 32 + koff) : z;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        acc0[rt] = mfma16(a0[u], b[u][rt], acc0[rt]);
        acc1[rt] = mfma16(a1[u], b[u][rt], acc1[rt]);
      }
  }
}

template <int RT>
__device__ __forceinline__ void zero_acc(f32x4_t (&acc)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

// ---------------------------------------------------------------- dense
// Y[r][n] (=|+=) X[r][:] . W[n][:], r < R, n < N.  Block = 4 waves, one
// 16-feature strip each; grid.y covers rows in groups of 16*RT.
template <int RT, bool ADD>
__global__ void __launch_bounds__(256) k_mm(int R, int N, int nkt, const uint16_t* __restrict__ X,
                                            int ldx_, const uint4* __restrict__ Wp,
                                            float* __restrict__ Y, int ldy) {
  const int lane = threadIdx.x & 63;
  const int nt = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (nt * 16 >= N) return;
  const int r0 = blockIdx.y * 16 * RT;
  const uint16_t* xr[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int r = r0 + rt * 16 + (lane & 15);
    xr[rt] = r < R ? X + (size_t)r * ldx_ : nullptr;
  }
  f32x4_t acc[RT];
  zero_acc(acc);
  strip_mma<RT>(Wp + (size_t)nt * nkt * 64, nkt, xr, acc);
  const int n = nt * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int r = r0 + rt * 16 + (lane & 15);
    if (r >= R || n >= N) continue;
    float4* y = (float4*)(Y + (size_t)r * ldy + n);
    float4 v = make_float4(acc[rt][0], acc[rt][1], acc[rt][2], acc[rt][3]);
    if (ADD) {
      float4 o = *y;
      v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
    }
    *y = v;
  }
}

// ---------------------------------------------------------------- QKV + RoPE + KV append
// Wave task w < D/16: a (q or k) rotate-half pair of strips -- features
// f and f + dh/2 of one head -- so RoPE is applied in registers; task
// w >= D/16: a strip of v.  q goes to q_out (float32, rotated); k (rotated)
// and v go to the cache at the row's position (valid rows only).
template <int RT>
__global__ void __launch_bounds__(256) k_qkv_rope(int R, int C, int nh, int dh, int nkt,
                                                  const uint16_t* __restrict__ X,
                                                  const uint4* __restrict__ Wp,
                                                  const float2* __restrict__ rope,
                                                  const int32_t* __restrict__ row_pos,
                                                  const int32_t* __restrict__ row_valid,
                                                  uint16_t* __restrict__ cache, size_t seq_stride,
                                                  int cap, float* __restrict__ q_out) {
  const int lane = threadIdx.x & 63;
  const int D = nh * dh, half = dh / 2, tph = dh / 32;  // pair tasks per head and section
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n_pair = 2 * nh * tph, n_task = n_pair + D / 16;
  if (w >= n_task) return;
  const int r0 = blockIdx.y * 16 * RT;
  const uint16_t* xr[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    int r = r0 + rt * 16 + (lane & 15);
    xr[rt] = r < R ? X + (size_t)r * nkt * 32 : nullptr;
  }
  if (w < n_pair) {
    const int sec = w / (nh * tph), rest = w % (nh * tph);
    const int h = rest / tph, pt = rest % tph;
    const int t0 = (sec * D + h * dh) / 16 + pt, t1 = t0 + tph;
    f32x4_t a0[RT], a1[RT];
    zero_acc(a0);
    zero_acc(a1);
    strip2_mma<RT>(Wp + (size_t)t0 * nkt * 64, Wp + (size_t)t1 * nkt * 64, nkt, xr, a0, a1);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = r0 + rt * 16 + (lane & 15);
      if (r >= R) continue;
      const int valid = row_valid[r];
      const int pos = valid ? row_pos[r] : 0;
      const int b = r / C;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int i = pt * 16 + 4 * (lane >> 4) + t;  // < dh/2
        const float2 cs = rope[(size_t)pos * half + i];
        const float x0 = a0[rt][t], x1 = a1[rt][t];
        const float y0 = x0 * cs.x - x1 * cs.y, y1 = x1 * cs.x + x0 * cs.y;
        if (sec == 0) {
          q_out[(size_t)r * D + h * dh + i] = y0;
          q_out[(size_t)r * D + h * dh + i + half] = y1;
        } else if (valid) {
          uint16_t* kc = cache + (size_t)b * seq_stride + ((size_t)h * cap + pos) * dh;
          kc[i] = f2bf(y0);
          kc[i + half] = f2bf(y1);
        }
      }
    }
  } else {
    const int vt = w - n_pair;
    f32x4_t a[RT];
    zero_acc(a);
    strip_mma<RT>(Wp + (size_t)(2 * D / 16 + vt) * nkt * 64, nkt, xr, a);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = r0 + rt * 16 + (lane & 15);
      if (r >= R || !row_valid[r]) continue;
      const int pos = row_pos[r], b = r / C;
      const int f = vt * 16 + 4 * (lane >> 4);
      const int h = f / dh, d = f % dh;
      uint16_t* vc = cache + (size_t)b * seq_stride + ((size_t)(nh + h) * cap + pos) * dh + d;
      uint2 pk;
      pk.x = (uint32_t)f2bf(a[rt][0]) | ((uint32_t)f2bf(a[rt][1]) << 16);
      pk.y = (uint32_t)f2bf(a[rt][2]) | ((uint32_t)f2bf(a[rt][3]) << 16);
      *(uint2*)vc = pk;
    }
  }
}

// ---------------------------------------------------------------- top-k helper
// Router decision for one row, one lane per expert (E <= 64): lv = the
// float32 logit (lanes >= E ignored).  Every lane reads all E logits from
// LDS (broadcast reads, no cross-lane chains) and derives its rank --
// #{j : l_j > l_e or (l_j == l_e and j < e)}, i.e. larger logit first, equal
// logits to the lower id -- and its float32 softmax probability.  Lanes of
// rank < topk write ridx/rw[rank]; gap = l_(k) - l_(k+1) (0 when k == E).
// sc is 68 floats of wave-private, 16-byte aligned LDS.
__device__ __forceinline__ void lane_topk(float lv, int E, int topk, float* sc, int32_t* ridx,
                                          float* rw, float* gap, int32_t* ridx_out, int* sel,
                                          float* selw) {
  const int lane = threadIdx.x & 63;
  sc[lane] = lane < E ? lv : -INFINITY;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_s_waitcnt(0);
  float mx = -INFINITY;
  int rank = 0;
#pragma unroll
  for (int j4 = 0; j4 < 16; ++j4) {
    const float4 v = *(const float4*)(sc + 4 * j4);
    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 4 * j4 + q;
      if (j < E) {
        mx = fmaxf(mx, vv[q]);
        rank += (vv[q] > lv) || (vv[q] == lv && j < lane);
      }
    }
  }
  float se = 0.f;
#pragma unroll
  for (int j4 = 0; j4 < 16; ++j4) {
    const float4 v = *(const float4*)(sc + 4 * j4);
    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (4 * j4 + q < E) se += __expf(vv[q] - mx);
  }
  const float p = __expf(lv - mx) / se;
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
  if (lane < E && rank == topk - 1) sc[64] = lv;
  if (lane < E && rank == topk) sc[65] = lv;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_s_waitcnt(0);
  if (lane == 0 && gap) *gap = topk < E ? sc[64] - sc[65] : 0.f;
}

// ---------------------------------------------------------------- router + grouping
// Block = 16 rows x 64 experts (E <= 64): logits by MFMA, bias, float32
// softmax, top-k (larger logit first, equal -> lower id), k-th vs
// (k+1)-th gap.  The last block to finish groups the (row, slot) pairs by
// expert: cnt[e], off[e] (exclusive prefix), and per entry its row, slot
// and gate weight, rows ascending within an expert.
__global__ void __launch_bounds__(256) k_router(int R, int E, int topk, int nkt,
                                                const uint16_t* __restrict__ X,
                                                const uint4* __restrict__ Wp,
                                                const float* __restrict__ bias,
                                                int32_t* __restrict__ ridx, float* __restrict__ rw,
                                                float* __restrict__ rgap,
                                                int32_t* __restrict__ ridx_out,
                                                int32_t* __restrict__ counter,
                                                int32_t* __restrict__ cnt, int32_t* __restrict__ off,
                                                int32_t* __restrict__ ent_row,
                                                int32_t* __restrict__ ent_slot,
                                                float* __restrict__ ent_w) {
  __shared__ float lg[16][65];
  __shared__ int last;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 16;
  if (wv * 16 < E) {
    const uint16_t* xr[1];
    const int r = r0 + (lane & 15);
    xr[0] = r < R ? X + (size_t)r * nkt * 32 : nullptr;
    f32x4_t acc[1];
    zero_acc(acc);
    strip_mma<1>(Wp + (size_t)wv * nkt * 64, nkt, xr, acc);
#pragma unroll
    for (int t = 0; t < 4; ++t) lg[lane & 15][wv * 16 + 4 * (lane >> 4) + t] = acc[0][t];
  }
  __syncthreads();
  // one wave per 4 rows: lane = expert
  __shared__ __align__(16) float tsc[4][68];
  for (int rr = wv; rr < 16; rr += 4) {
    const int r = r0 + rr;
    if (r >= R) break;
    float lv = -INFINITY;
    if (lane < E) {
      lv = lg[rr][lane];
      if (bias) lv += bias[lane];
    }
    lane_topk(lv, E, topk, tsc[wv], ridx + (size_t)r * topk, rw + (size_t)r * topk,
              rgap ? rgap + r : nullptr, ridx_out ? ridx_out + (size_t)r * topk : nullptr,
              nullptr, nullptr);
  }
  // last block: group by expert
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = atomicAdd(counter, 1) == (int)gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  if (threadIdx.x == 0) *counter = 0;  // self-reset for the next launch
  const int e = threadIdx.x;
  int c = 0;
  if (e < E)
    for (int x = 0; x < R * topk; ++x) c += ridx[x] == e;
  // exclusive prefix over experts (E <= 64: wave 0 holds all)
  __shared__ int sc[64];
  if (e < 64) sc[e] = e < E ? c : 0;
  __syncthreads();
  if (e < E) {
    int o = 0;
    for (int x = 0; x < e; ++x) o += sc[x];
    cnt[e] = c;
    off[e] = o;
    int t = o;
    for (int x = 0; x < R * topk; ++x)
      if (ridx[x] == e) {
        ent_row[t] = x / topk;
        ent_slot[t] = x % topk;
        ent_w[t] = rw[x];
        ++t;
      }
  }
}

// ---------------------------------------------------------------- MoE
// Gate/up of the routed experts (blockIdx.y = e < E: entries off[e]..+cnt[e])
// and of a dense SwiGLU over all rows (blockIdx.y == E, width SI, the shared
// experts as one SwiGLU -- or the draft FFN).  Wave = one 16-wide tile of
// the intermediate dimension for up to 64 entries (blockIdx.z chunk).
// act[entry][i] = bf16(silu(g) * u) (routed, row stride I); act_sh[r][i]
// (dense, row stride SI).
template <int RT>
__device__ __forceinline__ void gu_body(const uint4* __restrict__ G, const uint4* __restrict__ U,
                                        int nkt, const uint16_t* __restrict__ X, int ldx_,
                                        const int32_t* rows, int t0, int cnt, int it,
                                        uint16_t* __restrict__ act, int lda) {
  const int lane = threadIdx.x & 63;
  const uint16_t* xr[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int t = t0 + rt * 16 + (lane & 15);
    xr[rt] = t < cnt ? X + (size_t)(rows ? rows[t] : t) * ldx_ : nullptr;
  }
  f32x4_t ag[RT], au[RT];
  zero_acc(ag);
  zero_acc(au);
  strip2_mma<RT>(G, U, nkt, xr, ag, au);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int t = t0 + rt * 16 + (lane & 15);
    if (t >= cnt) continue;
    const int i = it * 16 + 4 * (lane >> 4);
    uint2 pk;
    pk.x = (uint32_t)f2bf(silu(ag[rt][0]) * au[rt][0]) |
           ((uint32_t)f2bf(silu(ag[rt][1]) * au[rt][1]) << 16);
    pk.y = (uint32_t)f2bf(silu(ag[rt][2]) * au[rt][2]) |
           ((uint32_t)f2bf(silu(ag[rt][3]) * au[rt][3]) << 16);
    *(uint2*)(act + (size_t)t * lda + i) = pk;
  }
}

__global__ void __launch_bounds__(256) k_moe_gu(int R, int E, int I, int SI, int nkt,
                                                const uint16_t* __restrict__ X,
                                                const uint4* __restrict__ egu, size_t e_stride,
                                                const uint4* __restrict__ sgu,
                                                const int32_t* __restrict__ cnt,
                                                const int32_t* __restrict__ off,
                                                const int32_t* __restrict__ ent_row,
                                                uint16_t* __restrict__ act,
                                                uint16_t* __restrict__ act_sh) {
  const int it = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int e = blockIdx.y;
  const int t0 = blockIdx.z * 64;
  const bool dense = e == E;
  const int width = dense ? SI : I;
  if (it * 16 >= width) return;
  const int n = dense ? R : cnt[e];
  if (t0 >= n) return;
  const uint4 *G, *U;
  const int32_t* rows;
  uint16_t* out;
  int lda;
  if (dense) {
    G = sgu + (size_t)it * nkt * 64;
    U = sgu + (size_t)(SI / 16 + it) * nkt * 64;
    rows = nullptr;
    out = act_sh;
    lda = SI;
  } else {
    const uint4* base = egu + (size_t)e * e_stride;
    G = base + (size_t)it * nkt * 64;
    U = base + (size_t)(I / 16 + it) * nkt * 64;
    rows = ent_row + off[e];
    out = act + (size_t)off[e] * I;
    lda = I;
  }
  if (n - t0 <= 16)
    gu_body<1>(G, U, nkt, X, nkt * 32, rows, t0, n, it, out, lda);
  else
    gu_body<4>(G, U, nkt, X, nkt * 32, rows, t0, n, it, out, lda);
}

// Down projection.  Routed (blockIdx.y = e < E): for each entry t of
// expert e, slot[(row*(k+1) + slot)][n] = w_t * (Wd_e[n] . act[t]).  Dense
// (blockIdx.y == E): slot[(r*(k+1) + k)][n] = Wsd[n] . act_sh[r].
template <int RT>
__device__ __forceinline__ void down_body(const uint4* __restrict__ A, int nkt,
                                          const uint16_t* __restrict__ act, int lda, int t0,
                                          int cnt, int nt, const int32_t* er, const int32_t* es,
                                          const float* ew, int topk, int H,
                                          float* __restrict__ slot) {
  const int lane = threadIdx.x & 63;
  const uint16_t* xr[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int t = t0 + rt * 16 + (lane & 15);
    xr[rt] = t < cnt ? act + (size_t)t * lda : nullptr;
  }
  f32x4_t acc[RT];
  zero_acc(acc);
  strip_mma<RT>(A, nkt, xr, acc);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int t = t0 + rt * 16 + (lane & 15);
    if (t >= cnt) continue;
    const int row = er ? er[t] : t;
    const int sl = er ? es[t] : topk;
    const float w = er ? ew[t] : 1.f;
    float4* dst = (float4*)(slot + ((size_t)row * (topk + 1) + sl) * H + nt * 16 + 4 * (lane >> 4));
    *dst = make_float4(w * acc[rt][0], w * acc[rt][1], w * acc[rt][2], w * acc[rt][3]);
  }
}

__global__ void __launch_bounds__(256) k_moe_down(int R, int E, int topk, int H, int I, int SI,
                                                  const uint16_t* __restrict__ act,
                                                  const uint16_t* __restrict__ act_sh,
                                                  const uint4* __restrict__ edn, size_t e_stride,
                                                  const uint4* __restrict__ sdn,
                                                  const int32_t* __restrict__ cnt,
                                                  const int32_t* __restrict__ off,
                                                  const int32_t* __restrict__ ent_row,
                                                  const int32_t* __restrict__ ent_slot,
                                                  const float* __restrict__ ent_w,
                                                  float* __restrict__ slot) {
  const int nt = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (nt * 16 >= H) return;
  const int e = blockIdx.y;
  const int t0 = blockIdx.z * 64;
  const bool dense = e == E;
  const int n = dense ? R : cnt[e];
  if (t0 >= n) return;
  if (dense) {
    const uint4* A = sdn + (size_t)nt * (SI / 32) * 64;
    if (n - t0 <= 16)
      down_body<1>(A, SI / 32, act_sh, SI, t0, n, nt, nullptr, nullptr, nullptr, topk, H, slot);
    else
      down_body<4>(A, SI / 32, act_sh, SI, t0, n, nt, nullptr, nullptr, nullptr, topk, H, slot);
  } else {
    const int o = off[e];
    const uint4* A = edn + (size_t)e * e_stride + (size_t)nt * (I / 32) * 64;
    if (n - t0 <= 16)
      down_body<1>(A, I / 32, act + (size_t)o * I, I, t0, n, nt, ent_row + o, ent_slot + o,
                   ent_w + o, topk, H, slot);
    else
      down_body<4>(A, I / 32, act + (size_t)o * I, I, t0, n, nt, ent_row + o, ent_slot + o,
                   ent_w + o, topk, H, slot);
  }
}

// h[r] += slot[r][k] (dense) + sum_{j<k} slot[r][j]; then RMSNorm of the
// new h with gain g -> xin (bf16, product input) and/or yf (float32).
// One block per row.  slot may be NULL (no MoE contribution to add).
__global__ void __launch_bounds__(256) k_combine_norm(int H, int topk,
                                                      const float* __restrict__ slot,
                                                      float* __restrict__ h,
                                                      const float* __restrict__ g, float eps,
                                                      float* __restrict__ yf,
                                                      uint16_t* __restrict__ xin) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  float* hr = h + (size_t)r * H;
  float ss = 0.f;
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    float v = hr[j];
    if (slot) {
      const float* s = slot + (size_t)r * (topk + 1) * H + j;
      float add = s[(size_t)topk * H];
      for (int x = 0; x < topk; ++x) add += s[(size_t)x * H];
      v += add;
      hr[j] = v;
    }
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float rinv = rsqrtf(ss / (float)H + eps);
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    const float y = hr[j] * rinv * g[j];
    if (yf) yf[(size_t)r * H + j] = y;
    if (xin) xin[(size_t)r * H + j] = f2bf(y);
  }
}

// ---------------------------------------------------------------- LM head
// Block = 64 vocabulary rows (4 strips) x up to 16*RT rows; per row it
// records the best logit, its id (lowest on ties) and the second best.
template <int RT>
__global__ void __launch_bounds__(256) k_lm_mfma(int R, int V, int nkt,
                                                 const uint16_t* __restrict__ X,
                                                 const uint4* __restrict__ Wp,
                                                 float* __restrict__ logits, size_t ldl,
                                                 float* __restrict__ pv, int32_t* __restrict__ pi,
                                                 float* __restrict__ p2) {
  __shared__ float bv[4][16 * RT], sv[4][16 * RT];
  __shared__ int bi[4][16 * RT];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int nt = blockIdx.x * 4 + wv;
  const int r0 = blockIdx.y * 16 * RT;
  const uint16_t* xr[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = r0 + rt * 16 + (lane & 15);
    xr[rt] = r < R ? X + (size_t)r * nkt * 32 : nullptr;
  }
  f32x4_t acc[RT];
  zero_acc(acc);
  const bool live = nt * 16 < V;
  if (live) strip_mma<RT>(Wp + (size_t)nt * nkt * 64, nkt, xr, acc);
  const int v0 = nt * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = r0 + rt * 16 + (lane & 15);
    float b1 = -INFINITY, b2 = -INFINITY;
    int id = 1 << 30;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int v = v0 + t;
      const float x = (live && v < V) ? acc[rt][t] : -INFINITY;
      if (logits && r < R && live && v < V) logits[(size_t)r * ldl + v] = x;
      if (x > b1) {
        b2 = b1;
        b1 = x;
        id = v;
      } else if (x > b2) {
        b2 = x;
      }
    }
    // merge the 4 lanes that hold the same row (lane, lane^16, lane^32, lane^48)
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
      bv[wv][rt * 16 + lane] = b1;
      sv[wv][rt * 16 + lane] = b2;
      bi[wv][rt * 16 + lane] = id;
    }
  }
  __syncthreads();
  if (threadIdx.x < 16 * RT) {
    const int rr = threadIdx.x, r = r0 + rr;
    if (r < R) {
      float b1 = bv[0][rr], b2 = sv[0][rr];
      int id = bi[0][rr];
      for (int x = 1; x < 4; ++x) {
        const float ob1 = bv[x][rr], ob2 = sv[x][rr];
        const int oid = bi[x][rr];
        if (ob1 > b1 || (ob1 == b1 && oid < id)) {
          b2 = fmaxf(b1, ob2);
          b1 = ob1;
          id = oid;
        } else {
          b2 = fmaxf(b2, ob1);
        }
      }
      const size_t o = (size_t)r * gridDim.x + blockIdx.x;
      pv[o] = b1;
      pi[o] = id;
      p2[o] = b2;
    }
  }
}

// one row of embeddings/vision -> h (float32) and its RMSNorm -> xin (bf16)
__global__ void __launch_bounds__(256) k_embed_norm(int C, int H, int V,
                                                    const int32_t* __restrict__ row_valid,
                                                    const int32_t* __restrict__ row_tok,
                                                    const uint16_t* __restrict__ embed,
                                                    const uint16_t* __restrict__ vision,
                                                    int vis_ld, int vis_off,
                                                    const float* __restrict__ g, float eps,
                                                    float* __restrict__ h,
                                                    uint16_t* __restrict__ xin,
                                                    int32_t* __restrict__ status) {
  extern __shared__ float sm[];
  __shared__ float red[16];
  const int r = blockIdx.x;
  load_input_row<true>(r, C, H, V, row_valid[r], row_tok, embed, vision, vis_ld, vis_off, sm,
                       status);
  float ss = 0.f;
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    h[(size_t)r * H + j] = sm[j];
    ss += sm[j] * sm[j];
  }
  ss = block_sum(ss, red);
  const float rinv = rsqrtf(ss / (float)H + eps);
  for (int j = threadIdx.x; j < H; j += blockDim.x) xin[(size_t)r * H + j] = f2bf(sm[j] * rinv * g[j]);
}

}  // namespace mtp
