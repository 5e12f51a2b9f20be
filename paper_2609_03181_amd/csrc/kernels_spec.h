// Greedy acceptance and the committed-token cache update.
#pragma once
#include "common.h"

namespace mtp {

// Acceptance equation: m = longest prefix with draft_s == verify_s;
// commit = [draft_1..draft_m, verify_{m+1}], padded with -1 to K+1.
__global__ void k_accept(int B, int K, const int32_t* __restrict__ draft,
                         const int32_t* __restrict__ verify, int32_t* __restrict__ accept_len,
                         int32_t* __restrict__ commit) {
  int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int32_t* d = draft + (size_t)b * K;
  const int32_t* v = verify + (size_t)b * (K + 1);
  int m = 0;
  while (m < K && d[m] == v[m]) ++m;
  int32_t* c = commit + (size_t)b * (K + 1);
  for (int s = 0; s < m; ++s) c[s] = d[s];
  c[m] = v[m];
  for (int s = m + 1; s <= K; ++s) c[s] = -1;
  accept_len[b] = m;
}

// Commit of the m+1 rows: length update only (their K/V already sit at
// their absolute positions; rows past the new length are dropped by the
// length itself).  Finished sequences are frozen.  An acceptance length
// outside [0, K] sets MTP_ERANGE and leaves the sequence unchanged.
__global__ void k_commit(int B, int K, const int32_t* __restrict__ accept_len,
                         const int32_t* __restrict__ commit, int32_t* __restrict__ kv_len,
                         int32_t* __restrict__ n_rows, int32_t* __restrict__ row_pos,
                         int32_t* __restrict__ pending, int32_t* __restrict__ next_tok,
                         const int32_t* __restrict__ max_new, int32_t* __restrict__ out_tok,
                         int max_out, int32_t* __restrict__ n_out, int32_t* __restrict__ status) {
  int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int limit = max_new ? min(max_new[b], max_out) : max_out;
  int no = n_out[b];
  if (no >= limit) return;
  int m = accept_len[b];
  if (m < 0 || m > K) {
    set_status(status, MTP_ERANGE);
    return;
  }
  const int32_t* c = commit + (size_t)b * (K + 1);
  int old = kv_len[b];
  kv_len[b] = old + m + 1;
  n_rows[b] = m + 1;
  row_pos[b] = old;
  pending[b] = c[m];
  for (int s = 0; s <= m; ++s) next_tok[(size_t)b * (K + 1) + s] = c[s];
  int take = min(m + 1, limit - no);
  for (int s = 0; s < take; ++s) out_tok[(size_t)b * max_out + no + s] = c[s];
  n_out[b] = no + take;
}

// End of prefill: step state for the first step.
__global__ void k_prefill_state(int B, int K, int P, const int32_t* __restrict__ tok_last,
                                int32_t* __restrict__ kv_len, int32_t* __restrict__ draft_len,
                                int32_t* __restrict__ next_tok, int32_t* __restrict__ n_rows,
                                int32_t* __restrict__ row_pos, int32_t* __restrict__ pending,
                                int32_t* __restrict__ out_tok, int max_out,
                                int32_t* __restrict__ n_out) {
  int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int t = tok_last[b];
  kv_len[b] = P;
  draft_len[b] = P - 1;
  next_tok[(size_t)b * (K + 1)] = t;
  n_rows[b] = 1;
  row_pos[b] = P - 1;
  pending[b] = t;
  if (max_out > 0) {
    out_tok[(size_t)b * max_out] = t;
    n_out[b] = 1;
  } else {
    n_out[b] = 0;
  }
}

// Benchmark harness: forced draft tokens from a per-step table.
__global__ void k_override(int B, int K, const int32_t* __restrict__ table, int n_steps,
                           int32_t* __restrict__ step_ctr, int32_t* __restrict__ draft) {
  int s = *step_ctr;
  if (s < 0 || s >= n_steps) s = 0;
  for (int i = threadIdx.x; i < B * K; i += blockDim.x) draft[i] = table[(size_t)s * B * K + i];
  __syncthreads();
  if (threadIdx.x == 0) *step_ctr = (s + 1) % n_steps;
}

// dst[b][0..H) = src[row idx[b]] (idx NULL: row b)
__global__ void k_copy_rows(int B, int H, const int32_t* __restrict__ idx,
                            const float* __restrict__ src, float* __restrict__ dst, size_t dst_ld) {
  int b = blockIdx.x;
  const float* s = src + (size_t)(idx ? idx[b] : b) * H;
  for (int j = threadIdx.x; j < H; j += blockDim.x) dst[(size_t)b * dst_ld + j] = s[j];
}

// routes of one prefill chunk (stage [L][B*C][k], row b*C+i) into the
// prefill layout out [L][B][n_rows][k] at rows c0+i
__global__ void k_scatter_routes(int L, int B, int C, int k, int n_rows, int c0,
                                 const int32_t* __restrict__ stage, int32_t* __restrict__ out) {
  const size_t n = (size_t)L * B * C * k;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(e % k);
    const size_t r = e / k;
    const int i = (int)(r % C), b = (int)((r / C) % B), l = (int)(r / ((size_t)C * B));
    out[(((size_t)l * B + b) * n_rows + c0 + i) * k + t] = stage[e];
  }
}

}  // namespace mtp
