// Straightforward VALU kernels: the float32 path of every op and the
// first correct bf16 path.  One wave per output feature, lanes split the
// reduction, rows processed in register blocks of RB.
#pragma once
#include "common.h"

namespace mtp {

constexpr int RB = 8;  // rows per register block

// Y[r][n] (=|+=) sum_k X[r][k] W[n][k] for r < R, n < N; K % 4 == 0.
// X is at product-input precision (row stride ldx); Y float32 (row stride ldy).
template <bool BF, bool ADD>
__global__ void __launch_bounds__(256) k_linear(int R, int N, int K,
                                                const typename St<BF>::T* __restrict__ X, int ldx,
                                                const typename St<BF>::T* __restrict__ W,
                                                float* __restrict__ Y, int ldy) {
  using S = St<BF>;
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const typename S::T* w = W + (size_t)n * K;
  for (int r0 = 0; r0 < R; r0 += RB) {
    float acc[RB];
#pragma unroll
    for (int q = 0; q < RB; ++q) acc[q] = 0.f;
    for (int k = lane * 4; k < K; k += 256) {
      float w0 = S::ld(w, k), w1 = S::ld(w, k + 1), w2 = S::ld(w, k + 2), w3 = S::ld(w, k + 3);
#pragma unroll
      for (int q = 0; q < RB; ++q) {
        if (r0 + q < R) {
          const typename S::T* x = X + (size_t)(r0 + q) * ldx + k;
          acc[q] += w0 * S::ld(x, 0) + w1 * S::ld(x, 1) + w2 * S::ld(x, 2) + w3 * S::ld(x, 3);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < RB; ++q) {
      float s = wave_sum(acc[q]);
      if (lane == 0 && r0 + q < R) {
        float* y = Y + (size_t)(r0 + q) * ldy + n;
        if (ADD) *y += s;
        else *y = s;
      }
    }
  }
}

// Decode attention, one block (256 threads) per (head, row): q (float32,
// RoPE applied) against keys 0..pos of its sequence, scale 1/sqrt(dh),
// softmax in float32 (running max over 256-key chunks), output at
// product-input precision.  Invalid rows write zeros.
template <bool BF>
__global__ void __launch_bounds__(256) k_attn(int C, int nh, int dh, const float* __restrict__ q,
                                              const typename St<BF>::T* __restrict__ cache,
                                              size_t seq_stride, int cap,
                                              const int32_t* __restrict__ row_pos,
                                              const int32_t* __restrict__ row_valid, float scale,
                                              typename St<BF>::T* __restrict__ out) {
  using S = St<BF>;
  __shared__ float qs[256];
  __shared__ float ps[256];
  __shared__ float red[16];
  __shared__ float accs[256];
  const int hh = blockIdx.x, r = blockIdx.y, t = threadIdx.x;
  const int D = nh * dh;
  typename S::T* o = out + (size_t)r * D + hh * dh;
  if (!row_valid[r]) {
    for (int j = t; j < dh; j += 256) S::st(o, j, 0.f);
    return;
  }
  const int pos = row_pos[r], b = r / C;
  const typename S::T* Kc = cache + (size_t)b * seq_stride + (size_t)(0 * nh + hh) * cap * dh;
  const typename S::T* Vc = cache + (size_t)b * seq_stride + (size_t)(1 * nh + hh) * cap * dh;
  if (t < dh) qs[t] = q[(size_t)r * D + hh * dh + t];
  __syncthreads();
  const int groups = 256 / dh;  // dh in {64, 128}
  const int d = t % dh, g = t / dh;
  float acc = 0.f, m_run = -INFINITY, l_run = 0.f;
  const int n_keys = pos + 1;
  for (int j0 = 0; j0 < n_keys; j0 += 256) {
    int j = j0 + t;
    float s = -INFINITY;
    if (j < n_keys) {
      const typename S::T* kr = Kc + (size_t)j * dh;
      float a = 0.f;
      for (int e = 0; e < dh; ++e) a += qs[e] * S::ld(kr, e);
      s = a * scale;
    }
    float m_new = fmaxf(m_run, block_max(s, red));
    float p = (j < n_keys) ? __expf(s - m_new) : 0.f;
    ps[t] = p;
    float psum = block_sum(p, red);  // contains the barrier that publishes ps
    float corr = __expf(m_run - m_new);
    l_run = l_run * corr + psum;
    acc *= corr;
    int jn = min(256, n_keys - j0);
    for (int jj = g; jj < jn; jj += groups) acc += ps[jj] * S::ld(Vc, (size_t)(j0 + jj) * dh + d);
    m_run = m_new;
    __syncthreads();
  }
  accs[t] = acc;
  __syncthreads();
  if (t < dh) {
    float s = 0.f;
    for (int gg = 0; gg < groups; ++gg) s += accs[gg * dh + t];
    S::st(o, t, s / l_run);
  }
}

// Router, one wave per row: logits l_e = y . Wr[e] (+ bias_e) for e < E
// (E <= 64, one lane per expert), float32 softmax over all E, top-k by
// logit (higher first, equal -> lower id), gap = l_(k) - l_(k+1).
template <bool BF>
__global__ void __launch_bounds__(256) k_router(int R, int E, int topk, int H,
                                                const typename St<BF>::T* __restrict__ y,
                                                const typename St<BF>::T* __restrict__ Wr,
                                                const float* __restrict__ bias,
                                                int32_t* __restrict__ ridx, float* __restrict__ rw,
                                                float* __restrict__ rgap,
                                                int32_t* __restrict__ ridx_out) {
  using S = St<BF>;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= R) return;
  const typename S::T* yr = y + (size_t)r * H;
  float l = -INFINITY;
  if (lane < E) {
    const typename S::T* wr = Wr + (size_t)lane * H;
    float a = 0.f;
    for (int k = 0; k < H; ++k) a += S::ld(yr, k) * S::ld(wr, k);
    if (bias) a += bias[lane];
    l = a;
  }
  float mx = wave_max(l);
  float ex = lane < E ? __expf(l - mx) : 0.f;
  float sum = wave_sum(ex);
  float p = ex / sum;
  bool taken = lane >= E;
  float kth = 0.f;
  for (int j = 0; j <= topk && j < E; ++j) {
    // wave argmax of (l, -lane) over untaken lanes
    float v = taken ? -INFINITY : l;
    int id = taken ? 1 << 30 : lane;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      float ov = __shfl_xor(v, o, MTP_WAVE);
      int oi = __shfl_xor(id, o, MTP_WAVE);
      if (ov > v || (ov == v && oi < id)) {
        v = ov;
        id = oi;
      }
    }
    if (j == topk) {
      if (lane == 0 && rgap) rgap[r] = kth - v;
      break;
    }
    if (lane == id) taken = true;
    float pid = __shfl(p, id, MTP_WAVE);
    if (lane == 0) {
      ridx[(size_t)r * topk + j] = id;
      rw[(size_t)r * topk + j] = pid;
      if (ridx_out) ridx_out[(size_t)r * topk + j] = id;
    }
    kth = v;
  }
  if (topk >= E && lane == 0 && rgap) rgap[r] = 0.f;
}

// MoE gate/up: for row r and slot j < k (routed expert ridx[r][j], width
// I) or j == k (the S shared experts as one SwiGLU of width S*I):
//   act[r][j][i] = in(silu(Wg[i] . y_r) * (Wu[i] . y_r)).
// One wave per (i, r, j).
template <bool BF>
__global__ void __launch_bounds__(256) k_moe_gu(int R, int topk, int H, int I, int SI,
                                                const typename St<BF>::T* __restrict__ y,
                                                const int32_t* __restrict__ ridx,
                                                const typename St<BF>::T* __restrict__ egu,
                                                const typename St<BF>::T* __restrict__ sgu,
                                                typename St<BF>::T* __restrict__ act) {
  using S = St<BF>;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int slot = blockIdx.y % (topk + 1), r = blockIdx.y / (topk + 1);
  const bool shared = slot == topk;
  const int width = shared ? SI : I;
  if (i >= width || r >= R) return;
  const typename S::T *wg, *wu;
  if (shared) {
    wg = sgu + (size_t)i * H;
    wu = sgu + (size_t)(SI + i) * H;
  } else {
    int e = ridx[(size_t)r * topk + slot];
    wg = egu + ((size_t)e * 2 * I + i) * H;
    wu = egu + ((size_t)e * 2 * I + I + i) * H;
  }
  const typename S::T* yr = y + (size_t)r * H;
  float ag = 0.f, au = 0.f;
  for (int k = lane; k < H; k += 64) {
    float yv = S::ld(yr, k);
    ag += yv * S::ld(wg, k);
    au += yv * S::ld(wu, k);
  }
  ag = wave_sum(ag);
  au = wave_sum(au);
  if (lane == 0) S::st(act, ((size_t)r * (topk + 1) + slot) * SI + i, silu(ag) * au);
}

// MoE down + combine + residual: h[r][n] += Wsd[n] . act[r][k] +
// sum_j w_j * (Wd_{e_j}[n] . act[r][j]).  One wave per (n, r).
template <bool BF>
__global__ void __launch_bounds__(256) k_moe_down(int R, int topk, int H, int I, int SI,
                                                  const typename St<BF>::T* __restrict__ act,
                                                  const int32_t* __restrict__ ridx,
                                                  const float* __restrict__ rw,
                                                  const typename St<BF>::T* __restrict__ edn,
                                                  const typename St<BF>::T* __restrict__ sdn,
                                                  float* __restrict__ h) {
  using S = St<BF>;
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int r = blockIdx.y;
  if (n >= H) return;
  const typename S::T* ar = act + (size_t)r * (topk + 1) * SI;
  const typename S::T* ws = sdn + (size_t)n * SI;
  float sh = 0.f;
  for (int k = lane; k < SI; k += 64) sh += S::ld(ws, k) * S::ld(ar + (size_t)topk * SI, k);
  float tot = wave_sum(sh);
  for (int j = 0; j < topk; ++j) {
    int e = ridx[(size_t)r * topk + j];
    const typename S::T* wd = edn + ((size_t)e * H + n) * I;
    float a = 0.f;
    for (int k = lane; k < I; k += 64) a += S::ld(wd, k) * S::ld(ar + (size_t)j * SI, k);
    tot += rw[(size_t)r * topk + j] * wave_sum(a);
  }
  if (lane == 0) h[(size_t)r * H + n] += tot;
}

// Dense SwiGLU activation from gate/up projections: gu [R][2F] float32
// (gate then up) -> act [R][F] at product-input precision.
template <bool BF>
__global__ void k_swiglu(int R, int F, const float* __restrict__ gu,
                         typename St<BF>::T* __restrict__ act) {
  using S = St<BF>;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)R * F) return;
  size_t r = i / F, c = i - r * F;
  S::st(act, i, silu(gu[r * 2 * F + c]) * gu[r * 2 * F + F + c]);
}

// LM head, partial argmax: block (256 threads) covers 64 vocabulary rows;
// for each input row it records the best logit, its id (lowest on ties)
// and the second-best logit over those 64.  Optionally writes logits.
template <bool BF>
__global__ void __launch_bounds__(256) k_lm_partial(int R, int V, int H,
                                                    const typename St<BF>::T* __restrict__ x,
                                                    const typename St<BF>::T* __restrict__ W,
                                                    float* __restrict__ logits, size_t ldl,
                                                    float* __restrict__ pv, int32_t* __restrict__ pi,
                                                    float* __restrict__ p2) {
  using S = St<BF>;
  __shared__ float tile[64][65];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int v0 = blockIdx.x * 64;
  const int nblk = gridDim.x;
  for (int rg = 0; rg < R; rg += 64) {
    const int nr = min(64, R - rg);
    for (int vv = w; vv < 64; vv += 4) {
      const int v = v0 + vv;
      for (int r0 = 0; r0 < nr; r0 += RB) {
        float acc[RB];
#pragma unroll
        for (int q = 0; q < RB; ++q) acc[q] = 0.f;
        if (v < V) {
          const typename S::T* wr = W + (size_t)v * H;
          for (int k = lane; k < H; k += 64) {
            float wv = S::ld(wr, k);
#pragma unroll
            for (int q = 0; q < RB; ++q)
              if (r0 + q < nr) acc[q] += wv * S::ld(x, (size_t)(rg + r0 + q) * H + k);
          }
        }
#pragma unroll
        for (int q = 0; q < RB; ++q) {
          float s = wave_sum(acc[q]);
          if (lane == 0 && r0 + q < nr) tile[r0 + q][vv] = v < V ? s : -INFINITY;
        }
      }
    }
    __syncthreads();
    if (logits) {
      for (int e = threadIdx.x; e < nr * 64; e += 256) {
        int rr = e >> 6, vv = e & 63;
        if (v0 + vv < V) logits[(size_t)(rg + rr) * ldl + v0 + vv] = tile[rr][vv];
      }
    }
    if (threadIdx.x < nr) {
      int rr = threadIdx.x;
      float best = -INFINITY, second = -INFINITY;
      int bi = v0;
      for (int vv = 0; vv < 64; ++vv) {
        float s = tile[rr][vv];
        if (s > best) {
          second = best;
          best = s;
          bi = v0 + vv;
        } else if (s > second) {
          second = s;
        }
      }
      size_t o = (size_t)(rg + rr) * nblk + blockIdx.x;
      pv[o] = best;
      pi[o] = bi;
      p2[o] = second;
    }
    __syncthreads();
  }
}

// Final argmax over the partials of each row: (best, lowest id on ties,
// margin = best - second).  One block per row (argmax_row); output row r
// goes to tok[(r / per) * ostride + ooff + r % per].
__global__ void __launch_bounds__(256) k_argmax_final(int R, int nblk, const float* __restrict__ pv,
                                                      const int32_t* __restrict__ pi,
                                                      const float* __restrict__ p2, int per,
                                                      int ostride, int ooff,
                                                      int32_t* __restrict__ tok,
                                                      float* __restrict__ margin) {
  const int r = blockIdx.x;
  float bv, sv;
  const int bi = argmax_row(r, nblk, pv, pi, p2, &bv, &sv);
  if (threadIdx.x == 0) {
    const int b = r / per, i = r - b * per;
    const size_t o = (size_t)b * ostride + ooff + i;
    tok[o] = bi;
    if (margin) margin[o] = bv - sv;
  }
}

}  // namespace mtp
