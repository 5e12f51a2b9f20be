// Row bookkeeping, embeddings, RMSNorm, RoPE + KV append.
#pragma once
#include "common.h"

namespace mtp {

// Zeroes words [0, n) of a 16-byte-aligned region with the whole grid
// (16-byte stores, then the tail).
__device__ __forceinline__ void zero_words(int32_t* __restrict__ z, int n) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x, nt = gridDim.x * blockDim.x;
  for (int q = t; q < n / 4; q += nt) ((int4*)z)[q] = make_int4(0, 0, 0, 0);
  for (int q = (n / 4) * 4 + t; q < n; q += nt) z[q] = 0;
}

// Row r = b*C + i of a pass over B sequences with C rows each sits at
// position pos0[b] + off + i (pos0 NULL: off + i).  It is valid when
// i < nvalid[b] (nvalid NULL: all) and its position is inside the cache.
// head_row[b] (optional) receives the index of the last valid row.
__global__ void k_rows_setup(int B, int C, const int32_t* __restrict__ pos0, int off,
                             const int32_t* __restrict__ nvalid, int cap,
                             int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
                             int32_t* __restrict__ head_row, int32_t* __restrict__ status,
                             int32_t* __restrict__ zero = nullptr, int n_zero = 0) {
  int r = blockIdx.x * blockDim.x + threadIdx.x;
  // counters that later kernels of the call expect at zero (the workspace
  // is carved differently by calls with other row counts)
  zero_words(zero, n_zero);
  if (r >= B * C) return;
  int b = r / C, i = r - b * C;
  int p = (pos0 ? pos0[b] : 0) + off + i;
  int nv = nvalid ? nvalid[b] : C;
  if (nv < 0 || nv > C) {
    set_status(status, MTP_ECAPACITY);
    nv = nv < 0 ? 0 : C;
  }
  int valid = i < nv;
  if (valid && (p < 0 || p >= cap)) {
    set_status(status, MTP_ECAPACITY);
    valid = 0;
  }
  row_pos[r] = p;
  row_valid[r] = valid;
  if (head_row && i == (nv > 0 ? nv - 1 : 0)) head_row[b] = r;
}

// row_tok[b*C + i] = src[b*ld + off + i] for off + i < ld, else -1
__global__ void k_row_tokens(int B, int C, const int32_t* __restrict__ src, int ld, int off,
                             int32_t* __restrict__ row_tok) {
  int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= B * C) return;
  int b = r / C, i = r - b * C;
  row_tok[r] = off + i < ld ? src[(size_t)b * ld + off + i] : -1;
}

// Depth-1 draft rows (catch-up): row r = b*C + i at row_pos_in[b] + i,
// valid when i < n_rows[b] and inside the cache, token next_tok[b*C + i];
// head_row[b] = the last valid row.  Row (b, 0) also checks that the
// catch-up starts inside the valid base-form region and moves its end to
// row_pos_in[b] + n_rows[b].  zero[0..n_zero) is cleared as in
// k_rows_setup.
__global__ void k_draft_rows(int B, int C, const int32_t* __restrict__ row_pos_in,
                             const int32_t* __restrict__ n_rows,
                             const int32_t* __restrict__ next_tok, int cap,
                             int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
                             int32_t* __restrict__ head_row, int32_t* __restrict__ row_tok,
                             int32_t* __restrict__ draft_len, int32_t* __restrict__ status,
                             int32_t* __restrict__ zero, int n_zero) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  zero_words(zero, n_zero);
  if (r >= B * C) return;
  const int b = r / C, i = r - b * C;
  const int p0 = row_pos_in[b], p = p0 + i;
  int nv = n_rows[b];
  if (nv < 0 || nv > C) {
    set_status(status, MTP_ECAPACITY);
    nv = nv < 0 ? 0 : C;
  }
  int valid = i < nv;
  if (valid && (p < 0 || p >= cap)) {
    set_status(status, MTP_ECAPACITY);
    valid = 0;
  }
  row_pos[r] = p;
  row_valid[r] = valid;
  row_tok[r] = next_tok[(size_t)b * C + i];
  if (i == (nv > 0 ? nv - 1 : 0)) head_row[b] = r;
  if (i == 0) {
    if (p0 > draft_len[b]) set_status(status, MTP_ECAPACITY);
    draft_len[b] = p0 + n_rows[b];
  }
}

// Draft chain row of depth d >= 2 (one row per sequence): position
// row_pos_in[b] + n_rows[b] - 1 + (d - 1), token draft_tok[b*K + d - 2].
__global__ void k_chain_rows(int B, int d, int K, const int32_t* __restrict__ row_pos_in,
                             const int32_t* __restrict__ n_rows,
                             const int32_t* __restrict__ draft_tok, int cap,
                             int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
                             int32_t* __restrict__ head_row, int32_t* __restrict__ row_tok,
                             int32_t* __restrict__ status) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int p = row_pos_in[b] + n_rows[b] - 1 + (d - 1);
  int valid = 1;
  if (p < 0 || p >= cap) {
    set_status(status, MTP_ECAPACITY);
    valid = 0;
  }
  row_pos[b] = p;
  row_valid[b] = valid;
  head_row[b] = b;
  row_tok[b] = draft_tok[(size_t)b * K + d - 2];
}

// NV (float4 per lane of an H-row read by one wave) for n4 = H/256
#define MTP_NV_DISPATCH(n4, F)     \
  do {                             \
    if ((n4) <= 2) { F(2); }       \
    else if ((n4) <= 4) { F(4); }  \
    else if ((n4) <= 5) { F(5); }  \
    else { F(8); }                 \
  } while (0)

// FastMTP draft input of one row by one wave (bf16 model, H % 256 == 0,
// H <= 256*NV): x[0..H) = N_e(e), x[H..2H) = N_h(a) rounded to bf16, with
// e the embedding row (bf16; NULL: zero) and a the state row (float32;
// NULL: zero).  Every load of the row is issued before the two sums.
template <int NV>
__device__ __forceinline__ void draft_in_wave(int H, const uint16_t* __restrict__ e,
                                              const float* __restrict__ a,
                                              const float* __restrict__ ge,
                                              const float* __restrict__ gh, float eps,
                                              uint16_t* __restrict__ x) {
  const int lane = threadIdx.x & 63, n4 = H / 256;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 ev[NV], av[NV], gev[NV], ghv[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    ev[u] = av[u] = gev[u] = ghv[u] = z;
    if (u < n4) {
      const int j4 = u * 64 + lane;  // float4 index within the row
      if (e) {
        const uint2 q = ((const uint2*)e)[j4];
        ev[u] = make_float4(bf2f((uint16_t)q.x), bf2f((uint16_t)(q.x >> 16)),
                            bf2f((uint16_t)q.y), bf2f((uint16_t)(q.y >> 16)));
      }
      if (a) av[u] = ld_f4(a + j4 * 4);
      gev[u] = ld_f4(ge + j4 * 4);
      ghv[u] = ld_f4(gh + j4 * 4);
    }
  }
  float se = 0.f, sa = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    se += ev[u].x * ev[u].x + ev[u].y * ev[u].y + ev[u].z * ev[u].z + ev[u].w * ev[u].w;
    sa += av[u].x * av[u].x + av[u].y * av[u].y + av[u].z * av[u].z + av[u].w * av[u].w;
  }
  se = wave_sum(se);
  sa = wave_sum(sa);
  const float re = rsqrtf(se / (float)H + eps), ra = rsqrtf(sa / (float)H + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    if (u < n4) {
      const int j4 = u * 64 + lane;
      uint2 pe, pa;
      pe.x = (uint32_t)f2bf(ev[u].x * re * gev[u].x) | ((uint32_t)f2bf(ev[u].y * re * gev[u].y) << 16);
      pe.y = (uint32_t)f2bf(ev[u].z * re * gev[u].z) | ((uint32_t)f2bf(ev[u].w * re * gev[u].w) << 16);
      pa.x = (uint32_t)f2bf(av[u].x * ra * ghv[u].x) | ((uint32_t)f2bf(av[u].y * ra * ghv[u].y) << 16);
      pa.y = (uint32_t)f2bf(av[u].z * ra * ghv[u].z) | ((uint32_t)f2bf(av[u].w * ra * ghv[u].w) << 16);
      ((uint2*)x)[j4] = pe;
      ((uint2*)(x + H))[j4] = pa;
    }
  }
}

// k_draft_rows and the draft input of its rows in one launch (bf16 model):
// one 64-thread block per row r = b*C + i; state row a[b*a_ld + i*H].
// Same bookkeeping, checks and zeroing as k_draft_rows; x[r] (2H bf16) as
// k_draft_in.  Tokens outside the vocabulary set MTP_ETOKEN (zero row).
template <int NV>
__global__ void __launch_bounds__(64) k_draft_rows_in(
    int B, int C, const int32_t* __restrict__ row_pos_in, const int32_t* __restrict__ n_rows,
    const int32_t* __restrict__ next_tok, int cap, int H, int V,
    const uint16_t* __restrict__ embed, const float* __restrict__ a, size_t a_ld,
    const float* __restrict__ ge, const float* __restrict__ gh, float eps,
    int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
    int32_t* __restrict__ head_row, int32_t* __restrict__ row_tok,
    int32_t* __restrict__ draft_len, int32_t* __restrict__ status, int32_t* __restrict__ zero,
    int n_zero, uint16_t* __restrict__ x) {
  const int r = blockIdx.x, lane = threadIdx.x;
  zero_words(zero, n_zero);
  if (r >= B * C) return;
  const int b = r / C, i = r - b * C;
  const int p0 = row_pos_in[b], p = p0 + i, nr = n_rows[b];
  const int t = next_tok[(size_t)b * C + i];
  int nv = nr;
  if (nv < 0 || nv > C) nv = nv < 0 ? 0 : C;
  int valid = i < nv;
  if (valid && (p < 0 || p >= cap)) valid = 0;
  const bool bad = valid && (t < 0 || t >= V);
  if (lane == 0) {
    if (nr != nv || (i < nv && !valid)) set_status(status, MTP_ECAPACITY);
    if (bad) set_status(status, MTP_ETOKEN);
    row_pos[r] = p;
    row_valid[r] = valid;
    row_tok[r] = t;
    if (i == (nv > 0 ? nv - 1 : 0)) head_row[b] = r;
    if (i == 0) {
      if (p0 > draft_len[b]) set_status(status, MTP_ECAPACITY);
      draft_len[b] = p0 + nr;
    }
  }
  const uint16_t* e = (valid && !bad) ? embed + (size_t)t * H : nullptr;
  const float* ar = valid ? a + (size_t)b * a_ld + (size_t)i * H : nullptr;
  draft_in_wave<NV>(H, e, ar, ge, gh, eps, x + (size_t)r * 2 * H);
}

// k_chain_rows and the draft input of its rows in one launch (bf16 model):
// one 256-thread block per sequence; state row a[b*H].  The depth d-1
// token is first reduced from the LM head's nblk partials of row b
// (pv/pi/p2 as k_argmax_final reads them) and stored to
// draft_tok[b*K + d-2]; then wave 0 sets up the row and its draft input.
template <int NV>
__global__ void __launch_bounds__(256) k_chain_rows_in(
    int B, int d, int K, const int32_t* __restrict__ row_pos_in,
    const int32_t* __restrict__ n_rows, int nblk, const float* __restrict__ pv,
    const int32_t* __restrict__ pi, const float* __restrict__ p2,
    int32_t* __restrict__ draft_tok, int cap, int H, int V,
    const uint16_t* __restrict__ embed, const float* __restrict__ a,
    const float* __restrict__ ge, const float* __restrict__ gh, float eps,
    int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
    int32_t* __restrict__ head_row, int32_t* __restrict__ row_tok, int32_t* __restrict__ status,
    uint16_t* __restrict__ x) {
  __shared__ int tok_s;
  const int b = blockIdx.x, lane = threadIdx.x & 63;
  if (b >= B) return;
  const int tr = argmax_row(b, nblk, pv, pi, p2);  // valid in thread 0
  if (threadIdx.x == 0) {
    draft_tok[(size_t)b * K + d - 2] = tr;
    tok_s = tr;
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  const int p = row_pos_in[b] + n_rows[b] - 1 + (d - 1);
  const int t = tok_s;
  const int valid = p >= 0 && p < cap;
  const bool bad = valid && (t < 0 || t >= V);
  if (lane == 0) {
    if (!valid) set_status(status, MTP_ECAPACITY);
    if (bad) set_status(status, MTP_ETOKEN);
    row_pos[b] = p;
    row_valid[b] = valid;
    head_row[b] = b;
    row_tok[b] = t;
  }
  const uint16_t* e = (valid && !bad) ? embed + (size_t)t * H : nullptr;
  const float* ar = valid ? a + (size_t)b * H : nullptr;
  draft_in_wave<NV>(H, e, ar, ge, gh, eps, x + (size_t)b * 2 * H);
}

// Loads input row r (token embedding, or a vision row when the token is
// negative) as float32 into smem[0..H).  Vision row of (b, i):
// vision[((size_t)b*vis_ld + vis_off + i)*H].  Invalid rows and bad tokens
// give a zero row (bad tokens of valid rows also set MTP_ETOKEN).
template <bool BF>
__device__ __forceinline__ void load_input_row(int r, int C, int H, int V, int valid,
                                               const int32_t* row_tok,
                                               const typename St<BF>::T* embed,
                                               const typename St<BF>::T* vision, int vis_ld,
                                               int vis_off, float* smem, int32_t* status) {
  using S = St<BF>;
  int t = row_tok[r];
  const typename S::T* src = nullptr;
  if (!valid) {
  } else if (t >= 0 && t < V) {
    src = embed + (size_t)t * H;
  } else if (t < 0 && vision) {
    int b = r / C, i = r - b * C;
    src = vision + ((size_t)b * vis_ld + vis_off + i) * H;
  } else if (threadIdx.x == 0) {
    set_status(status, MTP_ETOKEN);
  }
  for (int j = threadIdx.x; j < H; j += blockDim.x) smem[j] = src ? S::ld(src, j) : 0.f;
  __syncthreads();
}

// h[r][:] = input row r (float32 residual stream)
template <bool BF>
__global__ void k_embed(int R, int C, int H, int V, const int32_t* __restrict__ row_valid,
                        const int32_t* __restrict__ row_tok,
                        const typename St<BF>::T* __restrict__ embed,
                        const typename St<BF>::T* __restrict__ vision, int vis_ld, int vis_off,
                        float* __restrict__ h, int32_t* __restrict__ status) {
  extern __shared__ float sm[];
  int r = blockIdx.x;
  load_input_row<BF>(r, C, H, V, row_valid[r], row_tok, embed, vision, vis_ld, vis_off, sm,
                     status);
  for (int j = threadIdx.x; j < H; j += blockDim.x) h[(size_t)r * H + j] = sm[j];
}

// Verify rows fused with their embedding: row r = b*(K+1) + i at
// kv_len[b] + i (valid inside the cache), token pending[b] (i = 0) or
// draft[b*K + i - 1]; h[r] = its embedding row (zero for invalid rows; a
// token outside the vocabulary sets MTP_ETOKEN).  One block per row;
// zero[0..n_zero) is cleared as in k_rows_setup.
template <bool BF>
__global__ void k_verify_rows(int B, int K, const int32_t* __restrict__ kv_len,
                              const int32_t* __restrict__ pending,
                              const int32_t* __restrict__ draft, int cap, int H, int V,
                              const typename St<BF>::T* __restrict__ embed,
                              int32_t* __restrict__ row_pos, int32_t* __restrict__ row_valid,
                              float* __restrict__ h, int32_t* __restrict__ status,
                              int32_t* __restrict__ zero, int n_zero) {
  using S = St<BF>;
  zero_words(zero, n_zero);
  const int C = K + 1, r = blockIdx.x;
  if (r >= B * C) return;  // blocks past the rows only clear counters
  const int b = r / C, i = r - b * C;
  const int p = kv_len[b] + i;
  const int valid = p >= 0 && p < cap;
  const int t = i == 0 ? pending[b] : draft[(size_t)b * K + i - 1];
  if (threadIdx.x == 0) {
    if (!valid) set_status(status, MTP_ECAPACITY);
    else if (t < 0 || t >= V) set_status(status, MTP_ETOKEN);
    row_pos[r] = p;
    row_valid[r] = valid;
  }
  const typename S::T* src = (valid && t >= 0 && t < V) ? embed + (size_t)t * H : nullptr;
  for (int j = threadIdx.x; j < H; j += blockDim.x) h[(size_t)r * H + j] = src ? S::ld(src, j) : 0.f;
}

// RMSNorm of x[src_row] (float32, row stride ldx) with gain g:
//   y = x * rsqrt(mean(x^2) + eps) * g
// written as float32 to yf[o] (optional) and at the product-input
// precision to yin[o] (optional, row stride ldin, column offset col).
// src_row = idx ? idx[o] : o.  One block per output row o.
template <bool BF>
__global__ void k_rmsnorm(int H, const float* __restrict__ x, int ldx,
                          const int32_t* __restrict__ idx, const float* __restrict__ g, float eps,
                          float* __restrict__ yf, int ldf, typename St<BF>::T* __restrict__ yin,
                          int ldin, int col) {
  __shared__ float red[16];
  using S = St<BF>;
  int o = blockIdx.x;
  int r = idx ? idx[o] : o;
  const float* xr = x + (size_t)r * ldx;
  float ss = 0.f;
  for (int j = threadIdx.x; j < H; j += blockDim.x) ss += xr[j] * xr[j];
  ss = block_sum(ss, red);
  float rinv = rsqrtf(ss / (float)H + eps);
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    float y = xr[j] * rinv * g[j];
    if (yf) yf[(size_t)o * ldf + j] = y;
    if (yin) S::st(yin, (size_t)o * ldin + col + j, y);
  }
}

// FastMTP draft input: x[r] = [N_e(e_r); N_h(a_r)] at product-input
// precision, e_r = input row r, a_r = state row (float32).  State row of
// (b, i) is a[(size_t)b*a_ld + i*H].  One block per row.
template <bool BF>
__global__ void k_draft_in(int C, int H, int V, const int32_t* __restrict__ row_valid,
                           const int32_t* __restrict__ row_tok,
                           const typename St<BF>::T* __restrict__ embed,
                           const typename St<BF>::T* __restrict__ vision, int vis_ld, int vis_off,
                           const float* __restrict__ a, size_t a_ld,
                           const float* __restrict__ ge, const float* __restrict__ gh, float eps,
                           typename St<BF>::T* __restrict__ x, int32_t* __restrict__ status) {
  extern __shared__ float sm[];
  __shared__ float red[16];
  using S = St<BF>;
  int r = blockIdx.x;
  int b = r / C, i = r - b * C;
  const int valid = row_valid[r];
  load_input_row<BF>(r, C, H, V, valid, row_tok, embed, vision, vis_ld, vis_off, sm, status);
  const float* ar = a + (size_t)b * a_ld + (size_t)i * H;
  float* sa_row = sm + H;  // state row (zero for invalid rows)
  for (int j = threadIdx.x; j < H; j += blockDim.x) sa_row[j] = valid ? ar[j] : 0.f;
  __syncthreads();
  float se = 0.f, sa = 0.f;
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    se += sm[j] * sm[j];
    sa += sa_row[j] * sa_row[j];
  }
  se = block_sum(se, red);
  sa = block_sum(sa, red);
  float re = rsqrtf(se / (float)H + eps), ra = rsqrtf(sa / (float)H + eps);
  typename S::T* xr = x + (size_t)r * 2 * H;
  for (int j = threadIdx.x; j < H; j += blockDim.x) {
    S::st(xr, j, sm[j] * re * ge[j]);
    S::st(xr, H + j, sa_row[j] * ra * gh[j]);
  }
}

// RoPE (rotate-half) on q and k of every valid row, then K/V append:
// qkv [R][3D] float32 (q, k, v blocks of D = nh*dh); q_out [R][D] float32;
// k/v stored at cache[(b*seq_stride) + ((c*nh + h)*cap + pos)*dh + j].
// rope[pos][i] = (cos, sin) of pos * theta^(-2i/dh), i < dh/2.
template <bool BF>
__global__ void k_rope_kv(int C, int nh, int dh, const float* __restrict__ qkv,
                          const float2* __restrict__ rope, const int32_t* __restrict__ row_pos,
                          const int32_t* __restrict__ row_valid,
                          typename St<BF>::T* __restrict__ cache, size_t seq_stride, int cap,
                          float* __restrict__ q_out) {
  using S = St<BF>;
  int r = blockIdx.x;
  int D = nh * dh, half = dh >> 1;
  const float* q = qkv + (size_t)r * 3 * D;
  const float* k = q + D;
  const float* v = k + D;
  int valid = row_valid[r];
  int pos = valid ? row_pos[r] : 0;
  int b = r / C;
  typename S::T* kc = cache + (size_t)b * seq_stride;
  for (int t = threadIdx.x; t < nh * half; t += blockDim.x) {
    int hh = t / half, i = t - hh * half;
    float2 cs = rope[(size_t)pos * half + i];
    int j0 = hh * dh + i, j1 = j0 + half;
    float q0 = q[j0], q1 = q[j1];
    q_out[(size_t)r * D + j0] = q0 * cs.x - q1 * cs.y;
    q_out[(size_t)r * D + j1] = q1 * cs.x + q0 * cs.y;
    if (valid) {
      float k0 = k[j0], k1 = k[j1];
      size_t kb = ((size_t)(0 * nh + hh) * cap + pos) * dh;
      size_t vb = ((size_t)(1 * nh + hh) * cap + pos) * dh;
      S::st(kc, kb + i, k0 * cs.x - k1 * cs.y);
      S::st(kc, kb + i + half, k1 * cs.x + k0 * cs.y);
      S::st(kc, vb + i, v[j0]);
      S::st(kc, vb + i + half, v[j1]);
    }
  }
}

__global__ void k_fill_i32(int32_t* p, int n, int32_t v) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace mtp
