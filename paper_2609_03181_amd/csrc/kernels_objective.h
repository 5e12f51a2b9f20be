// FastMTP draft-head objective, forward (Section "Draft-head objective",
// Eq. draft-loss and Eq. objective): the state shift between the depths of
// the training grid and the per-row loss terms.  The draft block and the
// LM head of each depth are the library's multi-row draft and head kernels.
#pragma once
#include "common.h"

namespace mtp {

// States of the draft rows p = c0 + i (i < n) at depth `depth`
// (state-shift equation): b_p at depth 1 and on prompt rows (p < n_prompt),
// u_prev[p - 1] (the previous depth's output of the row before) otherwise.
__global__ void k_obj_states(int c0, int H, int depth, int n_prompt, const float* __restrict__ b,
                             const float* __restrict__ u_prev, float* __restrict__ a) {
  const int i = blockIdx.x, p = c0 + i;
  const float* src = (depth == 1 || p < n_prompt) ? b + (size_t)p * H : u_prev + (size_t)(p - 1) * H;
  for (int j = threadIdx.x * 4; j < H; j += blockDim.x * 4)
    *(float4*)(a + (size_t)i * H + j) = ld_f4(src + j);
}

// Storage-type copies of n float32 rows (the LM-head input of b_{p+1})
template <bool BF>
__global__ void k_obj_rows_in(int H, const float* __restrict__ x, typename St<BF>::T* __restrict__ y) {
  const int r = blockIdx.x;
  for (int j = threadIdx.x; j < H; j += blockDim.x) St<BF>::st(y, (size_t)r * H + j, x[(size_t)r * H + j]);
}

// double sum over a 256-thread block in a fixed order (deterministic)
__device__ __forceinline__ double block_sum_d(double v, double* red /* 256 */) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const double t = red[0];
  __syncthreads();
  return t;
}

// Loss terms of draft row p = c0 + i (one block per row): with P = softmax
// of the draft logits lp[i], Q = softmax of the verifier logits lq[i] (of
// b_{p+1}) and the target x_{p+2}:
//   CE = lse(lp) - lp[x_{p+2}]
//   KL(Q||P) = sum_v q_v (lq_v - lp_v) - lse(lq) + lse(lp)
//   MSE = ||u_p - b_{p+1}||^2
// for loss rows (n_prompt <= p <= n_rows - 3), zeros otherwise.  Maxima in
// float32, exponentials in float32, every sum in float64.  terms: [rows][3].
__global__ void __launch_bounds__(256) k_obj_terms(int c0, int n_rows, int n_prompt, int V, int H,
                                                   const float* __restrict__ lp,
                                                   const float* __restrict__ lq,
                                                   const float* __restrict__ u,
                                                   const float* __restrict__ b,
                                                   const int32_t* __restrict__ tok,
                                                   float* __restrict__ terms,
                                                   int32_t* __restrict__ status) {
  __shared__ float redf[16];
  __shared__ double redd[256];
  const int i = blockIdx.x, p = c0 + i;
  float* out = terms + (size_t)p * 3;
  if (p < n_prompt || p > n_rows - 3) {
    if (threadIdx.x < 3) out[threadIdx.x] = 0.f;
    return;
  }
  const float* P = lp + (size_t)i * V;
  const float* Q = lq + (size_t)i * V;
  float mp = -INFINITY, mq = -INFINITY;
  for (int v = threadIdx.x; v < V; v += blockDim.x) {
    mp = fmaxf(mp, P[v]);
    mq = fmaxf(mq, Q[v]);
  }
  mp = block_max(mp, redf);
  mq = block_max(mq, redf);
  double sp = 0.0, sq = 0.0, sqd = 0.0;
  for (int v = threadIdx.x; v < V; v += blockDim.x) {
    const float pv = P[v], qv = Q[v];
    const double eq = (double)expf(qv - mq);
    sp += (double)expf(pv - mp);
    sq += eq;
    sqd += eq * ((double)qv - (double)pv);
  }
  double ss = 0.0;
  const float* ur = u + (size_t)p * H;
  const float* br = b + (size_t)(p + 1) * H;
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    const double d = (double)ur[j] - (double)br[j];
    ss += d * d;
  }
  sp = block_sum_d(sp, redd);
  sq = block_sum_d(sq, redd);
  sqd = block_sum_d(sqd, redd);
  ss = block_sum_d(ss, redd);
  if (threadIdx.x == 0) {
    const int t = tok[p + 2];
    const bool ok = t >= 0 && t < V;
    if (!ok) set_status(status, MTP_ETOKEN);
    const double lse_p = (double)mp + log(sp), lse_q = (double)mq + log(sq);
    out[0] = ok ? (float)(lse_p - (double)P[t]) : 0.f;
    out[1] = (float)(sqd / sq - lse_q + lse_p);
    out[2] = (float)ss;
  }
}

// loss[3(k-1) + j] = mean of terms[k-1][p][j] over the loss rows
// p = n_prompt..n_rows-3 (j: CE, KL, MSE), loss[3K] = Eq. objective:
// 0.85 sum_k a_k CE_k + 0.45 sum_k a_k KL_k + 0.45 sum_k a_k MSE_k with
// a_k = beta^(k-1) / sum_r beta^(r-1).  One wave per (depth, term), lanes
// over rows in order, then a fixed wave reduction; float64 throughout.
__global__ void __launch_bounds__(256) k_obj_loss(int K, int n_rows, int n_prompt, double beta,
                                                  const float* __restrict__ terms,
                                                  double* __restrict__ loss) {
  __shared__ double means[8 * 3];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = n_rows - 2 - n_prompt;
  for (int q = w; q < 3 * K; q += blockDim.x >> 6) {
    const int k = q / 3, j = q % 3;
    double s = 0.0;
    for (int p = n_prompt + lane; p <= n_rows - 3; p += 64)
      s += (double)terms[((size_t)k * n_rows + p) * 3 + j];
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, MTP_WAVE);
    if (lane == 0) means[q] = s / (double)n;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double norm = 0.0, pw = 1.0;
    for (int k = 0; k < K; ++k, pw *= beta) norm += pw;
    double L = 0.0;
    pw = 1.0;
    for (int k = 0; k < K; ++k, pw *= beta) {
      const double a = pw / norm;
      L += a * (0.85 * means[3 * k] + 0.45 * means[3 * k + 1] + 0.45 * means[3 * k + 2]);
    }
    for (int q = 0; q < 3 * K; ++q) loss[q] = means[q];
    loss[3 * K] = L;
  }
}

}  // namespace mtp
