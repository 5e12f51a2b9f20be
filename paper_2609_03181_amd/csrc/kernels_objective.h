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

// Running float32 maxima and float64 sums of one pass over a row of logits:
// sp = sum exp(p - mp), sq = sum exp(q - mq), sqd = sum exp(q - mq) (q - p),
// rescaled (factor exp(m_old - m_new) in float64) when a maximum grows.
struct ObjStats {
  float mp = -INFINITY, mq = -INFINITY;
  double sp = 0.0, sq = 0.0, sqd = 0.0;
  __device__ __forceinline__ void rescale(float np_, float nq_) {
    if (np_ > mp) {
      sp = mp == -INFINITY ? 0.0 : sp * exp((double)mp - (double)np_);
      mp = np_;
    }
    if (nq_ > mq) {
      const double f = mq == -INFINITY ? 0.0 : exp((double)mq - (double)nq_);
      sq *= f;
      sqd *= f;
      mq = nq_;
    }
  }
  // n logits of P and Q (the caller raised the maxima over them first)
  template <int N>
  __device__ __forceinline__ void add(const float (&pv)[N], const float (&qv)[N]) {
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const double eq = (double)expf(qv[j] - mq);
      sp += (double)expf(pv[j] - mp);
      sq += eq;
      sqd += eq * ((double)qv[j] - (double)pv[j]);
    }
  }
};

// Loss terms of draft row p = c0 + i (one block per row): with P = softmax
// of the draft logits lp[i], Q = softmax of the verifier logits lq[i] (of
// b_{p+1}) and the target x_{p+2}:
//   CE = lse(lp) - lp[x_{p+2}]
//   KL(Q||P) = sum_v q_v (lq_v - lp_v) - lse(lq) + lse(lp)
//   MSE = ||u_p - b_{p+1}||^2
// for loss rows (n_prompt <= p <= n_rows - 3), zeros otherwise.  Maxima in
// float32, exponentials in float32, every sum in float64.  terms: [rows][3].
// One pass over the two rows (16-byte loads, four of each row in flight per
// thread; with V not a multiple of 4, 4-byte loads): each thread keeps
// running maxima and sums rescaled to them, then the block combines the
// threads' sums at the row maxima.
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
  const int i = blockIdx.x, p = c0 + i, t0 = threadIdx.x, nt = blockDim.x;
  float* out = terms + (size_t)p * 3;
  if (p < n_prompt || p > n_rows - 3) {
    if (threadIdx.x < 3) out[threadIdx.x] = 0.f;
    return;
  }
  const float* P = lp + (size_t)i * V;
  const float* Q = lq + (size_t)i * V;
  ObjStats st;
  if (V % 4 == 0) {
    constexpr int U = 4;
    const float4* P4 = (const float4*)P;
    const float4* Q4 = (const float4*)Q;
    const int n4 = V / 4;
    for (int v0 = t0; v0 < n4; v0 += U * nt) {
      float pv[4 * U], qv[4 * U];
#pragma unroll
      for (int u_ = 0; u_ < U; ++u_) {
        // past the row: a large negative finite value in both rows (its
        // exponentials are 0 and its q - p is 0; the batch's first piece is
        // always in the row, so it never sets a maximum)
        const bool in = v0 + u_ * nt < n4;
        const float4 a = in ? P4[v0 + u_ * nt] : make_float4(-3e38f, -3e38f, -3e38f, -3e38f);
        const float4 c = in ? Q4[v0 + u_ * nt] : make_float4(-3e38f, -3e38f, -3e38f, -3e38f);
        pv[4 * u_] = a.x; pv[4 * u_ + 1] = a.y; pv[4 * u_ + 2] = a.z; pv[4 * u_ + 3] = a.w;
        qv[4 * u_] = c.x; qv[4 * u_ + 1] = c.y; qv[4 * u_ + 2] = c.z; qv[4 * u_ + 3] = c.w;
      }
      float bp = -INFINITY, bq = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4 * U; ++j) {
        bp = fmaxf(bp, pv[j]);
        bq = fmaxf(bq, qv[j]);
      }
      st.rescale(bp, bq);
      st.add(pv, qv);
    }
  } else {
    for (int v = t0; v < V; v += nt) {
      float pv[1] = {P[v]}, qv[1] = {Q[v]};
      st.rescale(pv[0], qv[0]);
      st.add(pv, qv);
    }
  }
  // the block's maxima, then each thread's sums at them
  const float mp = block_max(st.mp, redf), mq = block_max(st.mq, redf);
  const double fp = st.mp == -INFINITY ? 0.0 : exp((double)st.mp - (double)mp);
  const double fq = st.mq == -INFINITY ? 0.0 : exp((double)st.mq - (double)mq);
  double sp = st.sp * fp, sq = st.sq * fq, sqd = st.sqd * fq;
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
