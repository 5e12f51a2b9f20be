// Fused MoE sub-layer for up to 16 rows: router, gate/up + SwiGLU of the
// touched routed experts and of the shared experts, and the down projection
// added to the residual stream, in one persistent launch per layer.
//
// Why one launch: at decode sizes the three steps are separated by their
// dependency latency, not by bytes (the router moves 0.2 MB).  In one
// launch the shared experts' tiles stream while the router runs, the down
// weights are requested before the gate/up tiles they multiply are
// finished, and no launch drains between the steps.
//
// Arithmetic is that of k_s_router + k_s_gu_stream + k_s_down_split (same
// tile order per wave, same wave-order sums, same fixed-point down sums), so
// the results equal theirs bit for bit.
#pragma once
#include "kernels_small.h"

namespace mtp {

// Per-layer synchronisation words (int32, zero at launch; the verify and
// prefill row set-up kernels clear them with the other counters).  Every
// word that waves poll sits on a 128-byte line of its own, and the
// routing-ready flag is replicated: hundreds of waves polling one line
// saturate the memory channel that holds it, which stalls every weight
// stream that also reads through that channel.
constexpr int kMoeLine = 32;                  // int32 words per 128-byte line
constexpr int kMoeAbort = 0;                  // a bounded wait expired: waits give up (line 0)
constexpr int kMoeFlags = 16;                 // copies of the router-strip flags: lines 1..16,
                                              // strip i's flag at word i of each line
constexpr int kMoeDone = (1 + kMoeFlags) * kMoeLine;  // one line per expert (E routed, S shared)
constexpr int kMoeMaxBlocks = 512;            // grid limit (one h-read flag word per block)
constexpr int kMoeDownTiles = 28;             // down tiles a wave requests before its wait
// then the down-strip counters (sixteen words apart, two per line) and the
// per-block flags "done reading h" (plain stores: no counter that every
// block would update)
__host__ __device__ inline int moe_strip_ctr(int E, int S) { return kMoeDone + (E + S) * kMoeLine; }
__host__ __device__ inline int moe_normed(int E, int S, int H) {
  return moe_strip_ctr(E, S) + ((H / 16 * 16 + kMoeLine - 1) / kMoeLine) * kMoeLine;
}
constexpr int kMoeSyncWords = 160 * kMoeLine;  // per layer

// Entry capacity of one gate/up tile of the routed outputs: each expert's
// entries start at a multiple of 4, so that one 128-byte line of the
// tile-major layout holds entries of one expert only.
__host__ __device__ inline int moe_entry_cap(int R, int topk, int E) {
  const int n = R * topk;
  return n + 3 * (E < n ? E : n);
}

// fixed-point down contributions: one H-wide row per routed entry slot
// (moe_entry_cap) and per (shared expert, row)
__host__ __device__ inline size_t moe_part_rows(int R, int topk, int E, int S) {
  return (size_t)moe_entry_cap(R, topk, E) + (size_t)S * R;
}

__device__ __forceinline__ int ld_agent_i(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait of the calling wave until *ctr >= target (polls about every
// 0.1 us plus the load's own latency).  False when the launch's abort word
// is set or the wait outlived spin_max polls (it then sets the abort word
// and MTP_ESTALL): the caller goes on with invalid data so that every wave
// still exits.
__device__ __forceinline__ bool moe_wait(const int32_t* ctr, int target, int32_t* sync,
                                         int32_t* status, int spin_max) {
  for (int i = 0;; ++i) {
    if (__builtin_amdgcn_readfirstlane(ld_agent_i(ctr)) >= target) break;
    if (i >= spin_max) {
      if ((threadIdx.x & 63) == 0) {
        __hip_atomic_store(sync + kMoeAbort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        set_status(status, MTP_ESTALL);
      }
      return false;
    }
    if ((i & 15) == 15 && __builtin_amdgcn_readfirstlane(ld_agent_i(sync + kMoeAbort)) != 0)
      return false;
    __builtin_amdgcn_s_sleep(4);
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return true;
}

// Work items of one launch, in this order (item k belongs to block
// k % gridDim.x, and a block takes its items in increasing k):
//   [0, NRT)                 router strip i: logits of experts 16i..16i+15 for
//                            every row, the four waves = four K-quarters summed
//                            in order (k_s_router's arithmetic)
//   [NRT, NRT + NSH)         shared gate/up tile (16 features of the width-S*I SwiGLU)
//   [.., + nT * I/16)        routed gate/up tile (touched expert in ascending id, tile)
//   [.., + (S + nT) * H/64)  down: (expert, quad of 16-wide output strips), the
//                            shared experts first
// Every block first normalises the rows into LDS.  Each router strip sets
// its flag in every copy once its logits are stored; a block reaching its
// first item past the shared tiles waits for the flags of all strips in
// its copy and then derives the routing itself
// (top-k and the grouping of (row, slot) pairs by expert: identical in
// every block; the block holding the first routed item writes the routing
// outputs).  A down wave requests its strip's weight tiles, then waits for
// the gate/up tiles of its expert.  Every wait is on items of
// lower index, so the lowest unfinished item can always proceed once every
// block is resident: the host launches at most (resident blocks per CU) x
// (CUs) blocks, and each wait is bounded.
//
// Hand-off between blocks (see common.h): router logits, gate/up outputs
// and down contributions are stored with agent-scope (write-through) stores
// and published by agent-scope counters after vmem_release; logits and
// contributions are read back with agent-scope loads.  The gate/up outputs
// are read with
// ordinary loads: they are tile-major (act[tile][entry][16],
// act_sh[tile][16 rows][16]) with every 128-byte line written by one item
// only and read only after that item's counter was seen, so no L2 can hold
// a stale copy of a line when it is read.
//
// h: residual [R][H] (float32), read by every block for the RMSNorm at its
// start.  The last block of each down strip adds the strip's fixed-point
// total to h, after checking that every block has flagged itself past that
// read.
template <int MAXT>
__global__ void __launch_bounds__(256, 2) k_s_moe(
    int R, int H, int E, int topk, int I, int S, float* __restrict__ h,
    const float* __restrict__ g, float eps, const uint4* __restrict__ Wr,
    const float* __restrict__ bias, const uint4* __restrict__ egu, size_t egu_s,
    const uint4* __restrict__ sgu, const uint4* __restrict__ edn, size_t edn_s,
    const uint4* __restrict__ sdn, float* __restrict__ lg, uint16_t* __restrict__ act,
    uint16_t* __restrict__ act_sh, unsigned long long* __restrict__ part,
    int32_t* __restrict__ sync, int32_t* __restrict__ ridx_out, float* __restrict__ rgap_out,
    int32_t* __restrict__ status, int spin_max) {
  extern __shared__ __align__(16) uint16_t xs[];  // [R][max(H, I) + XPAD]
  __shared__ f32x4_t red[2 * 4 * 64];
  __shared__ __align__(16) float tsc[4][68];
  __shared__ float s_lg[SR_MAX][65];
  __shared__ int s_sel[SR_MAX * 8];
  __shared__ float s_selw[SR_MAX * 8];
  __shared__ uint32_t s_mask[64];
  __shared__ int s_cnt[64], s_off[64], s_touched[64];
  __shared__ int s_ent_row[SR_MAX * 8 + 3 * 64];
  __shared__ float s_ent_w[SR_MAX * 8 + 3 * 64];
  __shared__ int s_nt;

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = lane & 15, koff = 8 * (lane >> 4);
  const int nkt = H / 32, per = nkt / 4, ldl = H + XPAD;
  const int nI = I / 16, SI = S * I, nsh = SI / 16, nkd = I / 32;
  const int NRT = (E + 15) / 16, base_r = NRT + nsh, nstrip = H / 16;
  const int ecap = moe_entry_cap(R, topk, E);
  int32_t* done = sync + kMoeDone;             // expert x: done[x * kMoeLine], x < E + S
  int32_t* sctr = sync + moe_strip_ctr(E, S);  // strip nt: sctr[16 * nt]
  int32_t* normed = sync + moe_normed(E, S, H);  // [gridDim.x]

  // gate/up item jj (0-based after the router strips): gate and up strips,
  // expert (-1: shared) and 16-wide tile
  auto gu_ptrs = [&](int jj, const uint4*& G, const uint4*& U, int& e, int& it) {
    if (jj < nsh) {
      e = -1;
      it = jj;
      G = sgu + (size_t)it * nkt * 64;
      U = sgu + (size_t)(nsh + it) * nkt * 64;
    } else {
      const int q = jj - nsh;
      e = s_touched[q / nI];
      it = q % nI;
      const uint4* base = egu + (size_t)e * egu_s;
      G = base + (size_t)it * nkt * 64;
      U = base + (size_t)(nI + it) * nkt * 64;
    }
  };

  int k = blockIdx.x;
  // ---- RMSNorm of the rows into LDS (every block).  Each wave's first row
  // is loaded before the tiles of a first item that needs no routing are
  // requested, so the sum does not wait for those tiles.
  NormRow<MTP_NV(MAXT)> nr0;
  if (w < R) norm_row_load<MTP_NV(MAXT)>(H, h + (size_t)w * H, g, nr0);
  uint4 ag[MAXT], au[MAXT];
  if (k < NRT) {
    preload<MAXT>(Wr + (size_t)k * nkt * 64, w * per, per, ag, true);
  } else if (k < base_r) {
    const uint4 *G, *U;
    int e, it;
    gu_ptrs(k - NRT, G, U, e, it);
    preload<MAXT>(G, w * per, per, ag, true);
    preload<MAXT>(U, w * per, per, au, true);
  }
  if (w < R) norm_row_store<MTP_NV(MAXT)>(H, eps, nr0, xs + w * ldl);
  norm_rows_lds<MTP_NV(MAXT)>(R, H, h, g, eps, xs, ldl, true);
  __syncthreads();
  if (threadIdx.x == 0)  // this block is done reading h
    __hip_atomic_store(normed + blockIdx.x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  if (k < NRT) {
    // ---- router strip k
    const uint16_t* xrow = t < R ? xs + t * ldl : nullptr;
    f32x4_t acc = mma_pre<MAXT, (MAXT % 4 == 0 ? 4 : (MAXT % 5 == 0 ? 5 : MAXT))>(
        ag, w * per, per, xrow, f32x4_t{0.f, 0.f, 0.f, 0.f});
    acc = block_acc_sum<4>(acc, red);
    if (w == 0) {
      if (t < R) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = k * 16 + 4 * (lane >> 4) + q;
          if (e < E) st_agent(lg + (size_t)t * E + e, acc[q]);
        }
      }
      vmem_release();  // the strip's logits are stored: set its flag in every copy
      if (lane < kMoeFlags)
        __hip_atomic_store(sync + (1 + lane) * kMoeLine + k, 1, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    k += gridDim.x;
  }

  // ---- shared gate/up tiles before the routing is known, then the routing
  // (the run loop below handles both; ngu grows once the routing is known)
  bool pre = k < base_r && k == (int)blockIdx.x;  // ag/au hold item k's tiles
  bool have_rt = false;
  int ngu = base_r;  // gate/up items known so far (the shared ones)
  for (;;) {
    if (k >= base_r && !have_rt) {
      // ---- routing: wait for every strip's flag, then top-k and grouping
      if (w == 0) {
        const int32_t* fl = sync + (1 + blockIdx.x % kMoeFlags) * kMoeLine;
        for (int i = 0;; ++i) {
          const int f = lane < NRT ? ld_agent_i(fl + lane) : 1;
          if (__ballot(f == 0) == 0ull) break;
          if (i >= spin_max) {
            if (lane == 0) {
              __hip_atomic_store(sync + kMoeAbort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              set_status(status, MTP_ESTALL);
            }
            break;
          }
          if ((i & 15) == 15 && __builtin_amdgcn_readfirstlane(ld_agent_i(sync + kMoeAbort)))
            break;
          __builtin_amdgcn_s_sleep(4);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
      __syncthreads();
      for (int x = threadIdx.x; x < R * E; x += blockDim.x)
        s_lg[x / E][x % E] = ld_agent(lg + x);
      __syncthreads();
      const bool writer = k == base_r;  // one block publishes the routing outputs
      const float bl = (bias && lane < E) ? bias[lane] : 0.f;
      for (int r = w; r < R; r += 4) {
        const float lv = lane < E ? s_lg[r][lane] + bl : -INFINITY;
        lane_topk(lv, E, topk, tsc[w], s_sel + r * topk, s_selw + r * topk,
                  (writer && rgap_out) ? rgap_out + r : nullptr,
                  (writer && ridx_out) ? ridx_out + (size_t)r * topk : nullptr, nullptr,
                  nullptr);
      }
      __syncthreads();
      const int nent = R * topk;
      if (threadIdx.x < 64) s_mask[threadIdx.x] = 0u;
      __syncthreads();
      if (threadIdx.x < nent) atomicOr(&s_mask[s_sel[threadIdx.x]], 1u << (threadIdx.x / topk));
      __syncthreads();
      if (w == 0) {
        const int c = lane < E ? __popc(s_mask[lane]) : 0;
        const int cp = (c + 3) & ~3;  // entries of an expert start at a multiple of 4
        int pre_sum = cp;             // inclusive scan over the 64 experts
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int v = __shfl_up(pre_sum, d, MTP_WAVE);
          if (lane >= d) pre_sum += v;
        }
        s_off[lane] = pre_sum - cp;
        s_cnt[lane] = c;
        const uint64_t has = __ballot(c > 0);
        if (c > 0) s_touched[__popcll(has & ((1ull << lane) - 1ull))] = lane;
        if (lane == 0) s_nt = __popcll(has);
      }
      __syncthreads();
      if (threadIdx.x < nent) {
        const int x = threadIdx.x, e = s_sel[x], r = x / topk;
        const int tt = s_off[e] + __popc(s_mask[e] & ((1u << r) - 1u));
        s_ent_row[tt] = r;
        s_ent_w[tt] = s_selw[x];
      }
      __syncthreads();
      have_rt = true;
      ngu = base_r + s_nt * nI;
    }
    if (k >= ngu) break;
    // ---- a run of gate/up tiles (k_s_gu_stream's arithmetic): while the
    // block's next item is a gate/up tile known already, its tiles are
    // requested as this item's MFMAs free the registers
    if (!pre) {
      const uint4 *G, *U;
      int e, it;
      gu_ptrs(k - NRT, G, U, e, it);
      preload<MAXT>(G, w * per, per, ag, true);
      preload<MAXT>(U, w * per, per, au, true);
    }
    for (;;) {
      const uint4 *G, *U;
      int e, it;
      gu_ptrs(k - NRT, G, U, e, it);
      const int kn = k + gridDim.x;
      const bool more = kn < ngu;
      const uint4 *Gn = G, *Un = U;
      int en = 0, itn = 0;
      if (more) gu_ptrs(kn - NRT, Gn, Un, en, itn);
      int n = R, o = 0;
      if (e >= 0) {
        n = s_cnt[e];
        o = s_off[e];
      }
      const int row = t < n ? (e >= 0 ? s_ent_row[o + t] : t) : 0;
      const uint16_t* xrow = xs + row * ldl;
      f32x4_t cg = {0.f, 0.f, 0.f, 0.f}, cu = cg;
#pragma unroll
      for (int u = 0; u < MAXT; ++u) {
        if (u < per) {
          const uint4 b = ldx(xrow + (w * per + u) * 32 + koff);
          cg = mfma16(ag[u], b, cg);
          cu = mfma16(au[u], b, cu);
          if (more) {
            ag[u] = ld_tile(Gn + (size_t)(w * per + u) * 64 + lane, true);
            au[u] = ld_tile(Un + (size_t)(w * per + u) * 64 + lane, true);
          }
        }
      }
      cg = block_acc_sum<4>(cg, red);
      cu = block_acc_sum<4>(cu, red + 4 * 64);
      if (w == 0) {
        if (t < n) {
          uint2 pk;
          pk.x = (uint32_t)f2bf(silu(cg[0]) * cu[0]) | ((uint32_t)f2bf(silu(cg[1]) * cu[1]) << 16);
          pk.y = (uint32_t)f2bf(silu(cg[2]) * cu[2]) | ((uint32_t)f2bf(silu(cg[3]) * cu[3]) << 16);
          const unsigned long long v = (unsigned long long)pk.x | ((unsigned long long)pk.y << 32);
          uint16_t* dst = e < 0 ? act_sh + ((size_t)it * 16 + t) * 16
                                : act + ((size_t)it * ecap + o + t) * 16;
          __hip_atomic_store((unsigned long long*)(dst + 4 * (lane >> 4)), v, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        }
        vmem_release();
        if (lane == 0)
          __hip_atomic_fetch_add(done + (e >= 0 ? e : E + (it * 16) / I) * kMoeLine, 1,
                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      k = kn;
      __syncthreads();  // red is free for the next item
      if (!more) break;
    }
    pre = false;
  }

  // ---- down items: (virtual expert, quad of output strips), the shared
  // experts first, then the touched routed experts in ascending id (the
  // order their gate/up tiles finish in).  After the expert's gate/up tiles
  // are done, its activation rows are staged in LDS once; wave w computes
  // strip 4q + w from weight tiles it requested before the wait and stores
  // each entry's fixed-point contribution w * (Wd[n] . act) (k_s_down_split's
  // values) to part[slot][H]: slot = the entry (routed) or ecap + sx*R + row
  // (shared).  The strip's last contributor sums, per row, the slots of its
  // top-k experts and the shared experts -- an exact integer sum, so the
  // result does not depend on the order -- and adds it to h.
  const int nvirt = s_nt + S, nquad = (nstrip + 3) / 4;
  const int total = ngu + nvirt * nquad;
  const int lda = I + XPAD;  // staging rows alias xs (free once the gate/up items are done)
  if (k < total && w == 0) {
    // before merging any strip into h: every block has flagged that it read
    // h (checked once, long before the first merge; bounded wait)
    for (int i = 0;; ++i) {
      int mine = 1;
      for (int b = lane; b < (int)gridDim.x; b += 64) mine &= ld_agent_i(normed + b);
      if (__ballot(!mine) == 0ull) break;
      if (i >= spin_max) {
        if (lane == 0) {
          __hip_atomic_store(sync + kMoeAbort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          set_status(status, MTP_ESTALL);
        }
        break;
      }
      __builtin_amdgcn_s_sleep(4);
    }
  }
  for (; k < total; k += gridDim.x) {
    const int d = k - ngu;
    const int vv = d / nquad, q = d - (d / nquad) * nquad;
    const bool shared = vv < S;
    const int nt = 4 * q + w;  // this wave's output strip
    const bool live = nt < nstrip;
    int n = R, o = 0, e = -1;
    const uint4* A;
    const int32_t* ctr;
    if (!shared) {
      e = s_touched[vv - S];
      n = s_cnt[e];
      o = s_off[e];
      A = edn + (size_t)e * edn_s + (size_t)(live ? nt : 0) * nkd * 64;
      ctr = done + e * kMoeLine;
    } else {
      A = sdn + (size_t)(live ? nt : 0) * S * nkd * 64 + (size_t)vv * nkd * 64;
      ctr = done + (E + vv) * kMoeLine;
    }
    uint4 a[kMoeDownTiles];
#pragma unroll
    for (int u = 0; u < kMoeDownTiles; ++u)
      a[u] = (live && u < nkd) ? ld_tile(A + (size_t)u * 64 + lane, true) : make_uint4(0, 0, 0, 0);
    if (w == 0) moe_wait(ctr, nI, sync, status, spin_max);
    __syncthreads();
    for (int x = threadIdx.x; x < n * nI * 2; x += blockDim.x) {  // 16-byte halves of row tiles
      const int half = x & 1, rt = x >> 1, it = rt % nI, r = rt / nI;
      const uint16_t* src = shared ? act_sh + (((size_t)vv * nI + it) * 16 + r) * 16
                                   : act + ((size_t)it * ecap + o + r) * 16;
      *(uint4*)(xs + r * lda + it * 16 + 8 * half) = *(const uint4*)(src + 8 * half);
    }
    __syncthreads();
    if (live) {
      const uint16_t* xrow = xs + (t < n ? t : 0) * lda;
      const uint4 z = make_uint4(0, 0, 0, 0);
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < kMoeDownTiles; ++u)
        if (u < nkd) acc = mfma16(a[u], t < n ? ldx(xrow + u * 32 + koff) : z, acc);
      for (int kt = kMoeDownTiles; kt < nkd; ++kt)  // longer strips: the rest tile by tile
        acc = mfma16(ld_tile(A + (size_t)kt * 64 + lane, true),
                     t < n ? ldx(xrow + kt * 32 + koff) : z, acc);
      bool bad = false;
      if (t < n) {
        const size_t slot = shared ? (size_t)ecap + (size_t)vv * R + t : (size_t)(o + t);
        const float wt = shared ? 1.f : s_ent_w[o + t];
        unsigned long long* pp = part + slot * H + nt * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          __hip_atomic_store(pp + qq, (unsigned long long)fx32(wt * acc[qq], bad),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (bad) set_status(status, MTP_ERANGE);
      vmem_release();
      int last = 0;
      if (lane == 0)
        last = __hip_atomic_fetch_add(sctr + 16 * nt, 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) == nvirt - 1;
      last = __builtin_amdgcn_readfirstlane(last);
      if (last) {  // (the block's wave 0 saw every h-read flag before its first down item)
        for (int x = lane; x < R * 16; x += 64) {
          const int r = x >> 4, f = x & 15;
          long long sum = 0;
          for (int j = 0; j < topk; ++j) {
            const int ex = s_sel[r * topk + j];
            const int slot = s_off[ex] + __popc(s_mask[ex] & ((1u << r) - 1u));
            sum += (long long)__hip_atomic_load(part + (size_t)slot * H + nt * 16 + f,
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
          for (int sx = 0; sx < S; ++sx)
            sum += (long long)__hip_atomic_load(
                part + ((size_t)ecap + (size_t)sx * R + r) * H + nt * 16 + f, __ATOMIC_RELAXED,
                __HIP_MEMORY_SCOPE_AGENT);
          h[(size_t)r * H + nt * 16 + f] += (float)sum * 2.3283064365386963e-10f;  // 2^-32
        }
      }
    }
    __syncthreads();  // the staging rows are free for the next item
  }
}

}  // namespace mtp
