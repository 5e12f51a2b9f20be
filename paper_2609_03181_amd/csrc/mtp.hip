// C-ABI implementation of the MI355X FastMTP greedy speculative-decode
// step (declarations and contracts in include/mtp.h).
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>

#include "common.h"
#include "kernels_generic.h"
#include "kernels_rows.h"
#include "kernels_mfma.h"
#include "kernels_small.h"
#include "kernels_fused.h"
#include "kernels_objective.h"
#include "kernels_flash.h"
#include "kernels_gemm.h"
#include "kernels_spec.h"

// 16-entry chunks a routed MoE block takes when a pass has 8 or more row
// groups (each weight tile read once per block is applied to all of them).
#ifndef MTP_MOE_CPB
#define MTP_MOE_CPB 4
#endif

using namespace mtp;

// Matrices of a bf16 model repacked into MFMA operand tiles (see
// kernels_mfma.h); strides are in uint4 units.
struct Packed {
  uint4* base;
  const uint4 *wqkv, *wo, *router, *exp_gu, *exp_down, *sh_gu, *sh_down, *lm;
  const uint4 *d_eh, *d_qkv, *d_wo, *d_gu, *d_down;
  size_t wqkv_s, wo_s, router_s, exp_gu_s, exp_down_s, sh_gu_s, sh_down_s;
};

// Launch timing of one kernel class (measurement hook): launches of the
// class go through hipExtLaunchKernelGGL with a start/stop event pair,
// which the runtime stamps at the dispatch's start and end.
struct Timing {
  int kclass = 0, cap = 0, n = 0;
  hipEvent_t* ev = nullptr;  // [2 * cap]: start, stop per launch
};

struct mtp_ctx {
  mtp_config cfg;
  mtp_weights w;
  float2* rope;      // [max_ctx][head_dim/2] (cos, sin)
  int32_t* dstatus;  // status word of the calls without a workspace
  void* scratch;     // device address of this device's static scratch
  Packed pk;         // bf16 models only
  size_t pk_bytes;   // bytes of the packed copy
  int n_split;   // attention key splits ...
  int spl;       // ... of spl positions each (multiple of 64)
  int n_cu;      // compute units of the device the context was created on
  int moe_blocks;  // resident blocks of the fused small-batch MoE (0: three launches)
  Timing tm;
};

// Launch of kernel k on stream s; timed when its class kc is being timed.
template <typename... KA, typename... Args>
inline void launch_k(Timing* tm, int kc, void (*k)(KA...), dim3 grid, dim3 block, size_t shmem,
                     hipStream_t s, Args... args) {
  if (tm && tm->kclass == kc && tm->n < tm->cap) {
    const int i = tm->n++;
    hipExtLaunchKernelGGL(k, grid, block, (uint32_t)shmem, s, tm->ev[2 * i], tm->ev[2 * i + 1], 0,
                          static_cast<KA>(args)...);
  } else {
    k<<<grid, block, shmem, s>>>(static_cast<KA>(args)...);
  }
}

// Static scratch of moe_verify_step_static: the workspace of the callers
// that cannot allocate.  Each device the library runs on holds its own
// copy until the process ends.  Host code never passes the array's name to
// a kernel (on the host it is a stand-in, not a device address): it uses
// the per-device address hipGetSymbolAddress returns (scratch_addr).
constexpr size_t kScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // per device: address of `scratch`, once zero-filled

// Address of the current device's static scratch (looked up and
// zero-filled on the first call for the device; the caller synchronises).
mtp_status scratch_addr(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MTP_EHIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MTP_EHIP;
    k_fill_i32<<<1024, 256>>>((int32_t*)p, (int)(kScratchBytes / 4), 0);
    if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) return MTP_EHIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MTP_OK;
}

constexpr int kLmBlk = 64;  // vocabulary rows per LM-head block
constexpr int kDownSplit = 8;  // blocks per output strip of the small-batch MoE down
constexpr int kMoeSpinMax = 1 << 20;  // polls of a fused-MoE wait before it gives up
constexpr int kSlotRows = 64;   // passes of 17..64 rows: slot-form MoE down and split-K QKV
constexpr int kFlashRows = 64;  // prefill passes of at least this many rows per sequence use
                                // the flash-style attention
constexpr int kFlashChunk = 4;      // key tiles per chunk of the split prefill attention
constexpr int kFlashChunkWide = 8;  // the same with at least as many (row tile, head) blocks as CUs

// Blocks of the fused small-batch MoE that the device holds at once (its
// waits need every block resident), or 0 when the shape is outside what it
// covers or MTP_FUSED_MOE=0 selects the three-launch form.
int moe_resident_blocks(const mtp_config& c, int n_cu) {
  const int H = c.hidden;
  if (c.dtype != MTP_BF16 || c.moe_inter > H ||
      moe_normed(c.n_routed, c.n_shared, H) + kMoeMaxBlocks > kMoeSyncWords)
    return 0;
  const char* env = getenv("MTP_FUSED_MOE");
  if (env && env[0] == '0') return 0;
  int occ = 0;
  hipError_t e = hipErrorInvalidValue;
  const size_t lds = (size_t)SR_MAX * (H + XPAD) * 2;
#define MTP_OCC(M) \
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, k_s_moe<M>, 256, lds)
  MTP_MAXT_DISPATCH(H / 128, MTP_OCC);
#undef MTP_OCC
  if (e != hipSuccess || occ < 1) return 0;
  return occ * n_cu < kMoeMaxBlocks ? occ * n_cu : kMoeMaxBlocks;
}

inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace carve for B sequences x C rows.
struct Ws {
  int32_t* status;
  int32_t* counter;  // self-resetting grid counter (router grouping)
  int32_t *row_pos, *row_valid, *row_tok, *head_row, *tok_stage, *chain_pos;
  float *h, *bbuf, *qkv, *q, *rw, *rgap, *gu, *ustate, *pv, *p2, *margin_stage;
  int32_t *ridx, *pi, *route_stage;
  void *xin, *attn, *act, *xhead;
  // bf16 fast path
  float *part, *slot, *ent_w;
  int32_t *cnt, *off, *ent_row, *ent_slot, *touched, *n_touched, *att_ctr, *dn_ctr;
  int32_t* cbp;  // chunk-block prefix of the grouped MoE GEMMs' items [E + 2]
  float* gpart;  // K-split partials of the dense tiled products (more than 16 rows)
  unsigned long long* dn_part;  // MoE down split partials [kDownSplit][R][H], fixed point (R <= 16)
  float* lg;                    // router logits of the fused MoE [R][E] (R <= 16)
  int32_t* moe_sync;            // fused MoE: kMoeSyncWords per layer (inside the zeroed counters)
  uint16_t* act_sh;
  int n_ctr;  // entries of att_ctr (zeroed at the start of each call)
  size_t bytes;
};

// Blocks of k_verify_rows: one per row, at least enough that the counters
// it clears take 16 words per thread (the fused MoE's sync words are
// ~64K words at up to 16 rows)
inline int verify_rows_grid(int R, int n_ctr) {
  const int zb = (n_ctr + 256 * 16 - 1) / (256 * 16);
  return R > zb ? R : zb;
}

// K splits of a dense tiled product of R rows, N outputs and K inputs: with
// few tiles (64-row chunks x 128-wide N-blocks) the K range is split so that
// about 256 blocks run, with at least two K chunks per split; 1 with 256
// tiles or more.  (Aiming at 384 or 768 blocks measured no faster at
// batch 16 and 64, and more splits write and read more float32 partials.)
inline int dense_splits(int R, int N, int K) {
  const int tiles = ((R + kGemmM - 1) / kGemmM) * (N / kGemmN), nch = K / kGemmKC;
  if (tiles >= 256 || nch < 4) return 1;
  const int want = (256 + tiles - 1) / tiles;
  const int cps = std::max(2, (nch + want - 1) / want);
  return (nch + cps - 1) / cps;
}

// Floats of the K-split partials of the dense products (QKV, O, eh, draft
// FFN gate/up and down) of any pass of 17..R rows: S * rows * columns, the
// largest over the products; within a 64-row chunk count S is fixed, so
// the chunk's last row count is the largest.
inline size_t dense_part_floats(const mtp_config& c, size_t R) {
  if (c.dtype != MTP_BF16) return 0;
  const int H = c.hidden, D = c.n_heads * c.head_dim, F = c.draft_inter;
  const int shape[5][3] = {{3 * D, H, 3 * D}, {H, D, H}, {H, 2 * H, H}, {H, F, H}, {F, H, 2 * F}};
  size_t best = 0;
  for (size_t r0 = SR_MAX; r0 < R; r0 = (r0 / kGemmM + 1) * kGemmM) {
    const size_t r = std::min(R, (r0 / kGemmM + 1) * kGemmM);
    for (const auto& sh : shape) {
      const int S = dense_splits((int)r, sh[0], sh[1]);
      if (S > 1) best = std::max(best, (size_t)S * r * sh[2]);
    }
  }
  return best;
}

Ws carve(const mtp_config& c, int B, int C, void* base, int n_split) {
  const size_t R = (size_t)B * C;
  const size_t es = c.dtype == MTP_BF16 ? 2 : 4;
  if (n_split < 1) n_split = 1;
  const int H = c.hidden, D = c.n_heads * c.head_dim, k = c.top_k;
  const int SI = c.n_shared * c.moe_inter;
  const size_t nblk = (c.vocab + kLmBlk - 1) / kLmBlk;
  size_t off = 0;
  char* p = (char*)base;
  auto take = [&](size_t bytes) {
    void* r = p ? p + off : nullptr;
    off += align_up(bytes);
    return r;
  };
  Ws w{};
  w.status = (int32_t*)take(128);
  w.counter = (int32_t*)take(128);
  w.row_pos = (int32_t*)take(R * 4);
  w.row_valid = (int32_t*)take(R * 4);
  w.row_tok = (int32_t*)take(R * 4);
  w.head_row = (int32_t*)take((size_t)B * 4);
  w.tok_stage = (int32_t*)take(R * 4);
  w.chain_pos = (int32_t*)take((size_t)B * 4);
  w.h = (float*)take(R * H * 4);
  w.bbuf = (float*)take(R * H * 4);
  w.qkv = (float*)take(R * 3 * D * 4);
  w.q = (float*)take(R * D * 4);
  w.ridx = (int32_t*)take(R * k * 4);
  w.rw = (float*)take(R * k * 4);
  w.rgap = (float*)take(R * 4);
  w.gu = (float*)take(R * 2 * (size_t)c.draft_inter * 4);
  w.ustate = (float*)take((size_t)B * H * 4);
  w.pv = (float*)take(R * nblk * 4);
  w.pi = (int32_t*)take(R * nblk * 4);
  w.p2 = (float*)take(R * nblk * 4);
  w.margin_stage = (float*)take(R * 4);
  w.route_stage = (int32_t*)take(R * k * (size_t)c.n_layers * 4);
  w.xin = take(R * 2 * H * es);
  w.attn = take(R * D * es);
  size_t act_cols = (size_t)(k + 1) * SI;
  if ((size_t)c.draft_inter > act_cols) act_cols = c.draft_inter;
  if (c.dtype == MTP_BF16) act_cols = (size_t)k * c.moe_inter;  // routed entries only
  size_t act_bytes = R * act_cols * es;
  // The fused small-batch MoE runs on any pass of up to 16 rows -- also the
  // last, shorter chunk of a prefill carved for longer chunks -- so every
  // bf16 carve holds its buffers, sized for min(R, 16) rows.
  const bool fused_rows = c.dtype == MTP_BF16;
  const int R16 = R < SR_MAX ? (int)R : SR_MAX;
  if (fused_rows) {  // tile-major gate/up outputs of the fused MoE
    const size_t fb = (size_t)(c.moe_inter / 16) * moe_entry_cap(R16, k, c.n_routed) * 16 * 2;
    if (fb > act_bytes) act_bytes = fb;
  }
  w.act = take(act_bytes);
  w.xhead = take(R * H * es);
  if (c.dtype == MTP_BF16) {
    w.part = (float*)take(R * c.n_heads * (size_t)n_split * (c.head_dim + 2) * 4);
    w.slot = (float*)take(R * (k + 1) * (size_t)H * 4);
    w.ent_w = (float*)take(R * k * 4);
    w.cnt = (int32_t*)take((size_t)c.n_routed * 4);
    w.off = (int32_t*)take((size_t)c.n_routed * 4);
    w.ent_row = (int32_t*)take(R * k * 4);
    w.ent_slot = (int32_t*)take(R * k * 4);
    w.touched = (int32_t*)take((size_t)c.n_routed * 4);
    w.n_touched = (int32_t*)take(4);
    w.cbp = (int32_t*)take(((size_t)c.n_routed + 2) * 4);
    // attention split counters then MoE-down strip counters, one region
    const size_t n_sync = fused_rows ? (size_t)c.n_layers * kMoeSyncWords : 0;
    w.att_ctr = (int32_t*)take((R * c.n_heads + (size_t)H / 16 + n_sync) * 4);
    w.dn_ctr = w.att_ctr + R * c.n_heads;
    w.moe_sync = fused_rows ? w.dn_ctr + H / 16 : nullptr;
    w.n_ctr = (int)(R * c.n_heads + H / 16 + n_sync);
    size_t part_rows = (size_t)kDownSplit * R16;
    if (moe_part_rows(R16, k, c.n_routed, c.n_shared) > part_rows)
      part_rows = moe_part_rows(R16, k, c.n_routed, c.n_shared);
    w.dn_part = (unsigned long long*)take(part_rows * H * 8);
    const size_t shw = (size_t)(SI > c.draft_inter ? SI : c.draft_inter);
    size_t sh_bytes = R * shw * 2;
    if (fused_rows && (size_t)SI * 16 * 2 > sh_bytes) sh_bytes = (size_t)SI * 16 * 2;
    w.act_sh = (uint16_t*)take(sh_bytes);
    w.lg = (float*)take((size_t)R16 * c.n_routed * 4);
    const size_t gp = dense_part_floats(c, R);
    w.gpart = gp ? (float*)take(gp * 4) : nullptr;
  } else {
    w.part = w.slot = w.ent_w = nullptr;
    w.cnt = w.off = w.ent_row = w.ent_slot = w.touched = w.n_touched = w.att_ctr = nullptr;
    w.cbp = nullptr;
    w.act_sh = nullptr;
    w.lg = nullptr;
    w.moe_sync = nullptr;
    w.gpart = nullptr;
  }
  w.bytes = off;
  return w;
}

inline unsigned cdiv(size_t a, size_t b) { return (unsigned)((a + b - 1) / b); }

template <bool BF>
struct Model {
  using T = typename St<BF>::T;
  const mtp_config& c;
  const mtp_weights& w;
  const float2* rope;
  hipStream_t s;
  const Packed& pk;
  int n_split;
  int spl;
  Timing* tm;
  int n_cu;              // compute units of the device (persistent grids)
  int moe_blocks = 0;    // fused small-batch MoE: grid that is resident at once (0: off)
  bool prefill = false;  // prefill calls launch the prefill-tagged kernel instances
  int pos_end = 0;       // prefill passes: a bound on their rows' positions + 1 (0: the cache size)

  const T* wp(const void* p, size_t off_elems) const { return (const T*)p + off_elems; }

  // one pre-norm attention sub-layer: h += Wo attn(RMSNorm(h; g))
  void attn_sublayer(const Ws& ws, int B, int C, const float* g, const T* wqkv, const T* wo,
                     T* cache, size_t seq_stride) {
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim, D = nh * dh;
    k_rmsnorm<BF><<<R, 256, 0, s>>>(H, ws.h, H, nullptr, g, (float)c.rms_eps, nullptr, 0,
                                    (T*)ws.xin, H, 0);
    k_linear<BF, false><<<cdiv(3 * D, 4), 256, 0, s>>>(R, 3 * D, H, (const T*)ws.xin, H, wqkv,
                                                       ws.qkv, 3 * D);
    k_rope_kv<BF><<<R, 256, 0, s>>>(C, nh, dh, ws.qkv, rope, ws.row_pos, ws.row_valid, cache,
                                    seq_stride, c.max_ctx, ws.q);
    k_attn<BF><<<dim3(nh, R), 256, 0, s>>>(C, nh, dh, ws.q, cache, seq_stride, c.max_ctx,
                                           ws.row_pos, ws.row_valid,
                                           1.0f / sqrtf((float)dh), (T*)ws.attn);
    k_linear<BF, true><<<cdiv(H, 4), 256, 0, s>>>(R, H, D, (const T*)ws.attn, D, wo, ws.h, H);
  }

  // LM head + greedy argmax over nr rows of xhead; token of row o goes to
  // tok[(o / per) * ostride + ooff + o % per].
  void lm_head(const Ws& ws, int nr, float* logits, size_t ldl, int per, int ostride, int ooff,
               int32_t* tok, float* margin) {
    const int V = c.vocab, H = c.hidden;
    const T* W = (const T*)(c.tie_lm_head ? w.embed : w.lm_head);
    const unsigned nblk = cdiv(V, kLmBlk);
    k_lm_partial<BF><<<nblk, 256, 0, s>>>(nr, V, H, (const T*)ws.xhead, W, logits, ldl, ws.pv,
                                          ws.pi, ws.p2);
    k_argmax_final<<<nr, 256, 0, s>>>(nr, nblk, ws.pv, ws.pi, ws.p2, per, ostride, ooff,
                                               tok, margin);
  }

  // Verifier over B x C rows (row tokens and row setup already in ws).
  // b states go to hid (row stride H); LM head on every row (head_all)
  // or on ws.head_row only.
  // embedded: ws.h already holds the input rows (the caller fused the
  // embedding into its row setup)
  // layer_h (checks): h entering layer l at layer_h + l*R*H, the last
  // layer's output at layer_h + L*R*H
  void snap_h(float* layer_h, int l, int R) {
    if (layer_h)
      (void)hipMemcpyAsync(layer_h + (size_t)l * R * c.hidden, pk_h, (size_t)R * c.hidden * 4,
                           hipMemcpyDeviceToDevice, s);
  }
  const float* pk_h = nullptr;  // ws.h of the current call (for snap_h)

  void verifier(const Ws& ws, int B, int C, const T* vision, int vis_ld, int vis_off, T* kv,
                float* hid, bool head_all, int32_t* tok, int per, int ostride, float* logits,
                float* margin, int32_t* route_idx, float* route_gap, bool embedded = false,
                float* layer_h = nullptr) {
    pk_h = ws.h;
    if constexpr (BF) {
      verifier_mfma(ws, B, C, vision, vis_ld, vis_off, kv, hid, head_all, tok, per, ostride,
                    logits, margin, route_idx, route_gap, embedded, layer_h);
      return;
    }
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim, D = nh * dh;
    const int L = c.n_layers, E = c.n_routed, k = c.top_k, I = c.moe_inter;
    const int SI = c.n_shared * I;
    const size_t seq_stride = (size_t)2 * nh * c.max_ctx * dh;
    const size_t layer_stride = (size_t)B * seq_stride;
    if (!embedded)
      k_embed<BF><<<R, 256, H * sizeof(float), s>>>(R, C, H, c.vocab, ws.row_valid, ws.row_tok, (const T*)w.embed,
                                                  vision, vis_ld, vis_off, ws.h, ws.status);
    for (int l = 0; l < L; ++l) {
      snap_h(layer_h, l, R);
      attn_sublayer(ws, B, C, w.attn_norm + (size_t)l * H, wp(w.wqkv, (size_t)l * 3 * D * H),
                    wp(w.wo, (size_t)l * H * D), kv + (size_t)l * layer_stride, seq_stride);
      k_rmsnorm<BF><<<R, 256, 0, s>>>(H, ws.h, H, nullptr, w.ffn_norm + (size_t)l * H,
                                      (float)c.rms_eps, nullptr, 0, (T*)ws.xin, H, 0);
      k_router<BF><<<cdiv(R, 4), 256, 0, s>>>(
          R, E, k, H, (const T*)ws.xin, wp(w.router, (size_t)l * E * H),
          w.router_bias ? w.router_bias + (size_t)l * E : nullptr, ws.ridx, ws.rw,
          route_gap ? route_gap + (size_t)l * R : ws.rgap,
          route_idx ? route_idx + (size_t)l * R * k : nullptr);
      k_moe_gu<BF><<<dim3(cdiv(SI > I ? SI : I, 4), R * (k + 1)), 256, 0, s>>>(
          R, k, H, I, SI, (const T*)ws.xin, ws.ridx, wp(w.exp_gu, (size_t)l * E * 2 * I * H),
          wp(w.sh_gu, (size_t)l * 2 * SI * H), (T*)ws.act);
      k_moe_down<BF><<<dim3(cdiv(H, 4), R), 256, 0, s>>>(
          R, k, H, I, SI, (const T*)ws.act, ws.ridx, ws.rw, wp(w.exp_down, (size_t)l * E * H * I),
          wp(w.sh_down, (size_t)l * H * SI), ws.h);
    }
    snap_h(layer_h, L, R);
    k_rmsnorm<BF><<<R, 256, 0, s>>>(H, ws.h, H, nullptr, w.final_norm, (float)c.rms_eps, hid, H,
                                    nullptr, 0, 0);
    if (!tok) return;
    if (head_all) {
      k_rmsnorm<BF><<<R, 256, 0, s>>>(H, ws.h, H, nullptr, w.final_norm, (float)c.rms_eps,
                                      nullptr, 0, (T*)ws.xhead, H, 0);
      lm_head(ws, R, logits, c.vocab, per, ostride, 0, tok, margin);
    } else {
      k_rmsnorm<BF><<<B, 256, 0, s>>>(H, ws.h, H, ws.head_row, w.final_norm, (float)c.rms_eps,
                                      nullptr, 0, (T*)ws.xhead, H, 0);
      lm_head(ws, B, logits, c.vocab, 1, 1, 0, tok, margin);
    }
  }

  // Draft block over B x C rows with states a (row (b, i) at
  // a + b*a_ld + i*H) and inputs from ws.row_tok / vision.  With a head,
  // the last valid row of each sequence gives ws.ustate[b] (its u) and its
  // greedy token at tok[b*ostride + ooff].
  // xin_ready (bf16 model): the caller has written the draft input rows to
  // ws.xin already (row setup fused with the draft input)
  // defer_argmax (bf16 model): the head's token reduction is left to the
  // next depth's row setup
  // kv_only (no head): the block's K/V rows are all the caller needs, so
  // the bf16 block stops once they are appended (attention, O projection
  // and FFN outputs would go unread), the float32 one after its attention
  // sub-layer
  void draft(const Ws& ws, int B, int C, const float* a, size_t a_ld, const T* vision, int vis_ld,
             int vis_off, T* dkv, bool head, int32_t* tok, int ostride, int ooff, float* logits,
             size_t ldl, bool xin_ready = false, bool defer_argmax = false, bool kv_only = false) {
    if constexpr (BF) {
      draft_mfma(ws, B, C, a, a_ld, vision, vis_ld, vis_off, dkv, head, tok, ostride, ooff,
                 logits, ldl, xin_ready, defer_argmax, kv_only && !head);
      return;
    }
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim, D = nh * dh;
    const int F = c.draft_inter;
    const size_t seq_stride = (size_t)2 * nh * c.max_ctx * dh;
    k_draft_in<BF><<<R, 256, 2 * H * sizeof(float), s>>>(C, H, c.vocab, ws.row_valid, ws.row_tok, (const T*)w.embed,
                                                     vision, vis_ld, vis_off, a, a_ld, w.d_enorm,
                                                     w.d_hnorm, (float)c.rms_eps, (T*)ws.xin,
                                                     ws.status);
    k_linear<BF, false><<<cdiv(H, 4), 256, 0, s>>>(R, H, 2 * H, (const T*)ws.xin, 2 * H,
                                                   (const T*)w.d_eh_proj, ws.h, H);
    attn_sublayer(ws, B, C, w.d_attn_norm, (const T*)w.d_wqkv, (const T*)w.d_wo, dkv, seq_stride);
    if (kv_only && !head) return;
    k_rmsnorm<BF><<<R, 256, 0, s>>>(H, ws.h, H, nullptr, w.d_ffn_norm, (float)c.rms_eps, nullptr,
                                    0, (T*)ws.xin, H, 0);
    k_linear<BF, false><<<cdiv(2 * F, 4), 256, 0, s>>>(R, 2 * F, H, (const T*)ws.xin, H,
                                                       (const T*)w.d_gu, ws.gu, 2 * F);
    k_swiglu<BF><<<cdiv((size_t)R * F, 256), 256, 0, s>>>(R, F, ws.gu, (T*)ws.act);
    k_linear<BF, true><<<cdiv(H, 4), 256, 0, s>>>(R, H, F, (const T*)ws.act, F,
                                                  (const T*)w.d_down, ws.h, H);
    if (!head) return;
    k_rmsnorm<BF><<<B, 256, 0, s>>>(H, ws.h, H, ws.head_row, w.final_norm, (float)c.rms_eps,
                                    ws.ustate, H, (T*)ws.xhead, H, 0);
    lm_head(ws, B, logits, ldl, 1, ostride, ooff, tok, nullptr);
  }
  // ------------------------------------------------------------ bf16 MFMA path
  static int nw_for(int nkt) {
    if (nkt % 16 == 0 && nkt >= 128) return 16;
    if (nkt % 8 == 0 && nkt >= 64) return 8;
    return 4;
  }
  static unsigned groups(int R) { return (unsigned)((R + 15) / 16); }
  // grid of an XCD-ordered tiled launch for at most `items` work items
  static unsigned grid_xcd(size_t items) { return (unsigned)(cdiv(items, kXcd) * kXcd); }
  static size_t lds_rows(int R, int H) { return (size_t)(R < 16 ? R : 16) * (H + XPAD) * 2; }

  // Y (=|+=) X . W^T over R rows (16-row groups)
  // Dense tiled product of R > 16 rows (kernels_gemm.h), K split over
  // blocks when there are few tiles (then a reduce launch adds the splits)
  template <int MODE>
  void dense(const Ws& ws, int kc, int R, int N, int K, const uint16_t* X, int ldx,
             const uint4* Wp, const DenseOut& o) {
    const int S = dense_splits(R, N, K);
    launch_k(tm, kc, k_dense_gemm<MODE>, dim3(grid_xcd((size_t)cdiv(R, kGemmM) * (N / kGemmN) * S)),
             dim3(256), 0, s, R, N, K, X, ldx, Wp, S, ws.gpart, o);
    if (S > 1)
      launch_k(tm, kc, k_dense_reduce<MODE>,
               dim3(cdiv((size_t)R * (MODE == DG_QKV ? N / 8 : N / 4), 256)), dim3(256), 0, s, R, N,
               S, (const float*)ws.gpart, o);
  }

  void smm(const Ws& ws, int R, int N, int K, const uint16_t* X, int ldx_, const uint4* Wp,
           float* Y, int ldy, bool add) {
    // tiled GEMM (rows in LDS) beyond 16 rows, except the short products
    // (K <= 2560: O projection, eh) of decode-sized passes, where the
    // split-K form with one block per (strip, row group) measured faster
    if (R > SR_MAX && N % kGemmN == 0 && K % kGemmKC == 0 && (K > 2560 || R > 256)) {
      DenseOut o{};
      o.y = Y;
      o.ldy = ldy;
      if (add) dense<DG_ADD>(ws, 0, R, N, K, X, ldx_, Wp, o);
      else dense<DG_SET>(ws, 0, R, N, K, X, ldx_, Wp, o);
      return;
    }
    const int nkt = K / 32, nw = nw_for(nkt), per = nkt / nw;
    const dim3 g(cdiv(N, 16), groups(R));
#define MTP_SMM_T(NW, M)                                                                   \
  if (add) k_s_mm<NW, true, M><<<g, NW * 64, 0, s>>>(R, N, nkt, X, ldx_, Wp, Y, ldy);      \
  else k_s_mm<NW, false, M><<<g, NW * 64, 0, s>>>(R, N, nkt, X, ldx_, Wp, Y, ldy);
#define MTP_SMM(NW)                                   \
  if (per <= 4) { MTP_SMM_T(NW, 4) }                  \
  else if (per <= 10) { MTP_SMM_T(NW, 10) }           \
  else if (per <= 16) { MTP_SMM_T(NW, 16) }           \
  else { MTP_SMM_T(NW, 0) }
    if (nw == 16) { MTP_SMM(16) } else if (nw == 8) { MTP_SMM(8) } else { MTP_SMM(4) }
#undef MTP_SMM
#undef MTP_SMM_T
  }

  // Key splits for one call: enough blocks to fill the chip, splits of at
  // least 64 positions, at most the context's n_split.  The block target
  // (live blocks are fewer: splits past a sequence's keys exit) is 2048
  // for at most 256 (row group, head) pairs and 4096 above (measured: batch
  // 16 -- 160 pairs -- attention 40.4 us at 2048 against 45.9 at 4096;
  // batch 64 -- 640 pairs -- 151 us at 4096 against 192 at 2048).
  void splits_for(int blocks_per_split, int& ns, int& sp) const {
    const int target = blocks_per_split <= 256 ? 2048 : 4096;
    ns = (target + blocks_per_split - 1) / blocks_per_split;
    const int cap64 = (c.max_ctx + 63) / 64;
    if (ns > n_split) ns = n_split;
    if (ns > cap64) ns = cap64;
    if (ns < 1) ns = 1;
    sp = ((c.max_ctx + ns - 1) / ns + 63) / 64 * 64;
    ns = (c.max_ctx + sp - 1) / sp;
  }
  template <int DH, int NR>
  void sattn_launch(const Ws& ws, int B, int C, uint16_t* cache, size_t seq_stride) {
    const int ng = (C + NR - 1) / NR;
    int ns, sp;
    splits_for(B * ng * c.n_heads, ns, sp);
    launch_k(tm, MTP_KC_ATTN, k_s_attn<DH, NR>, dim3(ns, c.n_heads, B * ng), dim3(256), 0, s, C,
             c.n_heads, ns, sp, ws.q, cache, seq_stride, c.max_ctx, ws.row_pos, ws.row_valid,
             1.0f / sqrtf((float)DH), ws.part, ws.att_ctr, (uint16_t*)ws.attn);
  }
  // 128-dim heads: one kernel for every row count (groups of four rows),
  // so a row's result is the same in the verify pass (K+1 rows), the draft
  // passes, plain greedy decoding (one row) and prefill chunks of any size
  void sattn4(const Ws& ws, int B, int C, uint16_t* cache, size_t seq_stride) {
    const int ng = (C + 3) / 4;
    int ns, sp;
    splits_for(B * ng * c.n_heads, ns, sp);
    launch_k(tm, MTP_KC_ATTN, k_s_attn4<128>, dim3(ns, c.n_heads, B * ng), dim3(256), 0, s, C,
             c.n_heads, ns, sp, ws.q, cache, seq_stride, c.max_ctx, ws.row_pos, ws.row_valid,
             1.0f / sqrtf(128.f), ws.part, ws.att_ctr, (uint16_t*)ws.attn);
  }
  template <int DH>
  void sattn(const Ws& ws, int B, int C, uint16_t* cache, size_t seq_stride) {
    if (DH == 128 && prefill && C >= kFlashRows) {  // prefill passes: flash-style, both products on MFMA
      // The keys in chunks, run in parallel and merged by a second launch,
      // so no block walks more than a chunk's tiles (the causal rows of the
      // last row tiles would otherwise set the launch's length): chunks of
      // kFlashChunk tiles with fewer (row tile, head) blocks than compute
      // units, of kFlashChunkWide tiles with more (measured at 1,668 rows:
      // 5.78 ms unsplit, 5.59 ms in chunks of 8; at 768 rows, 120 blocks:
      // 3.01 ms in chunks of 4 against 3.12 in chunks of 2)
      const int nt = cdiv(C, 64);
      const int kt = cdiv(pos_end > 0 && pos_end < c.max_ctx ? pos_end : c.max_ctx, 64);
      const int fch = nt * c.n_heads * B < n_cu ? kFlashChunk : kFlashChunkWide;
      const int nch = cdiv(kt, fch);
      if (nch > 1 && nch <= n_split) {
        launch_k(tm, MTP_KC_ATTN, k_flash_prefill<128, true>, dim3(nt * nch, c.n_heads, B),
                 dim3(256), 0, s, C, c.n_heads, ws.q, cache, seq_stride, c.max_ctx, ws.row_pos,
                 ws.row_valid, 1.0f / sqrtf(128.f), (uint16_t*)ws.attn, nt, fch, nch, ws.part);
        launch_k(tm, MTP_KC_ATTN, k_attn_merge<128>, dim3(cdiv((size_t)B * C * c.n_heads, 4)),
                 dim3(256), 0, s, B * C, c.n_heads, fch, nch, (const float*)ws.part,
                 ws.row_pos, ws.row_valid, (uint16_t*)ws.attn);
        return;
      }
      launch_k(tm, MTP_KC_ATTN, k_flash_prefill<128>, dim3(nt, c.n_heads, B), dim3(256), 0, s, C,
               c.n_heads, ws.q, cache, seq_stride, c.max_ctx, ws.row_pos, ws.row_valid,
               1.0f / sqrtf(128.f), (uint16_t*)ws.attn, nt, 0, 0, (float*)nullptr);
      return;
    }
    if (DH == 128) sattn4(ws, B, C, cache, seq_stride);
    else if (C <= 1) sattn_launch<DH, 1>(ws, B, C, cache, seq_stride);
    else if (C <= 2) sattn_launch<DH, 2>(ws, B, C, cache, seq_stride);
    else if (C <= 4) sattn_launch<DH, 4>(ws, B, C, cache, seq_stride);
    else sattn_launch<DH, 8>(ws, B, C, cache, seq_stride);
  }

  // attention sub-layer: h += Wo attn(RMSNorm(h; g)).  With xg the
  // normalised rows are already in xg (bf16) and g is unused.  kv_only:
  // only the K/V rows appended to the cache are wanted (stops after QKV).
  void attn_mfma(const Ws& ws, int B, int C, const float* g, const uint16_t* xg,
                 const uint4* wqkv, const uint4* wo, uint16_t* cache, size_t seq_stride,
                 bool kv_only = false) {
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim, D = nh * dh;
    if (xg && R > kSlotRows) {  // tiled GEMM over the normalised rows
      DenseOut o{};
      o.C = C;
      o.nh = nh;
      o.dh = dh;
      o.cap = c.max_ctx;
      o.seq_stride = seq_stride;
      o.rope = rope;
      o.row_pos = ws.row_pos;
      o.row_valid = ws.row_valid;
      o.cache = cache;
      o.q_out = ws.q;
      dense<DG_QKV>(ws, MTP_KC_QKV, R, 3 * D, H, xg, H, wqkv, o);
    } else {
#define MTP_QKV(M)                                                                          \
  launch_k(tm, MTP_KC_QKV, (!xg && groups(R) == 1) ? k_s_qkv<M, true> : k_s_qkv<M, false>,   \
           dim3(D / 8, groups(R)), dim3(256),                                                 \
           xg ? 0 : lds_rows(R, H), s, R, C, H, nh, dh, ws.h, g, (float)c.rms_eps, xg, wqkv, \
           rope, ws.row_pos, ws.row_valid, cache, seq_stride, c.max_ctx, ws.q)
      MTP_MAXT_DISPATCH(H / 128, MTP_QKV);
#undef MTP_QKV
    }
    if (kv_only) return;
    if (dh == 128) sattn<128>(ws, B, C, cache, seq_stride);
    else sattn<64>(ws, B, C, cache, seq_stride);
    smm(ws, R, H, D, (const uint16_t*)ws.attn, D, wo, ws.h, H, true);
  }

  // LM head over nr rows of ws.xhead (bf16, normalised), greedy argmax
  // RMSNorm of n rows of ws.h-like x (rows idx[o], or o) by one wave each
  // (bf16 model)
  void norm_rows(int n, const float* x, const int32_t* idx, const float* g, float* yf,
                 uint16_t* yb) {
    const int H = c.hidden, n4 = H / 256;
    const float eps = (float)c.rms_eps;
#define MTP_NR(NV) k_norm_rows<NV><<<n, 64, 0, s>>>(H, x, idx, g, eps, yf, yb)
    MTP_NV_DISPATCH(n4, MTP_NR);
#undef MTP_NR
  }
  // LM-head partials per row (blocks of the launch lm_mfma makes for nr rows)
  unsigned lm_partials(int nr) const {
    return groups(nr) >= 4 ? cdiv(c.vocab, 128) : cdiv(cdiv(c.vocab, 16), 4);
  }
  // defer_argmax: the partials are left in ws.pv/pi/p2 for the next kernel
  void lm_mfma(const Ws& ws, int nr, float* logits, size_t ldl, int per, int ostride, int ooff,
               int32_t* tok, float* margin, bool defer_argmax = false) {
    const int V = c.vocab, H = c.hidden;
    const unsigned nblk = cdiv(cdiv(V, 16), 4);
    const unsigned G = groups(nr);
    unsigned nb = nblk;
    if (G >= 4) {  // many rows: the tiled GEMM, 128 (from 128 rows: 256) vocabulary rows x 64 rows per block
      const bool wide = nr >= 2 * kGemmM;
      nb = cdiv(V, wide ? 2 * kGemmN : kGemmN);
      DenseOut o{};
      o.logits = logits;
      o.ldl = ldl;
      o.pv = ws.pv;
      o.pi = ws.pi;
      o.p2 = ws.p2;
      launch_k(tm, MTP_KC_LM_HEAD, wide ? k_dense_gemm<DG_ARGMAX_W> : k_dense_gemm<DG_ARGMAX>,
               dim3(grid_xcd((size_t)cdiv(nr, kGemmM) * nb)), dim3(256), 0, s, nr, V, H,
               (const uint16_t*)ws.xhead, H, pk.lm, 1, (float*)nullptr, o);
    } else if (G >= 2) {
      launch_k(tm, MTP_KC_LM_HEAD, k_s_lm<2>, dim3(nblk, cdiv(G, 2)), dim3(256), 0, s, nr, V, H,
               (const uint16_t*)ws.xhead, pk.lm, logits, ldl, ws.pv, ws.pi, ws.p2,
               (const float*)nullptr, (const int32_t*)nullptr, (const float*)nullptr, 0.f,
               (float*)nullptr);
    } else {  // one row group; above 4 rows the rows are staged in LDS once per block
      const bool xl = nr > 4;
      launch_k(tm, MTP_KC_LM_HEAD, xl ? k_s_lm<1, true> : k_s_lm<1, false>, dim3(nblk, G),
               dim3(256), xl ? lds_rows(nr, H) : 0, s, nr, V, H, (const uint16_t*)ws.xhead, pk.lm,
               logits, ldl, ws.pv, ws.pi, ws.p2, (const float*)nullptr, (const int32_t*)nullptr,
               (const float*)nullptr, 0.f, (float*)nullptr);
    }
    if (!defer_argmax)
      k_argmax_final<<<nr, 256, 0, s>>>(nr, nb, ws.pv, ws.pi, ws.p2, per, ostride, ooff, tok,
                                        margin);
  }
  // RMSNorm (gain g) of nr rows of x (rows idx[o], or o; float32 copies to
  // yf when given) and the LM head on them.  Up to 4 rows in one launch:
  // every block of the head normalises the rows into LDS while its first
  // weight tiles load (its first block writes yf), so the norm costs no
  // launch of its own (measured: batch 1 922 -> 930 tokens/s); more rows:
  // norm_rows, then lm_mfma (at 16 rows every block normalising them all
  // measured slower: batch 16 18,217 -> 18,044).
  void head_norm(const Ws& ws, int nr, const float* x, const int32_t* idx, const float* g,
                 float* yf, float* logits, size_t ldl, int per, int ostride, int ooff,
                 int32_t* tok, float* margin, bool defer_argmax = false) {
    const int V = c.vocab, H = c.hidden;
    if (nr > 4) {
      norm_rows(nr, x, idx, g, yf, (uint16_t*)ws.xhead);
      lm_mfma(ws, nr, logits, ldl, per, ostride, ooff, tok, margin, defer_argmax);
      return;
    }
    const unsigned nblk = cdiv(cdiv(V, 16), 4);
    const float eps = (float)c.rms_eps;
#define MTP_HN(NV)                                                                            \
  launch_k(tm, MTP_KC_LM_HEAD, k_s_lm<1, true, NV>, dim3(nblk, 1), dim3(256), lds_rows(nr, H), \
           s, nr, V, H, (const uint16_t*)nullptr, pk.lm, logits, ldl, ws.pv, ws.pi, ws.p2, x,   \
           idx, g, eps, yf)
    MTP_NV_DISPATCH(H / 256, MTP_HN);
#undef MTP_HN
    if (!defer_argmax)
      k_argmax_final<<<nr, 256, 0, s>>>(nr, nblk, ws.pv, ws.pi, ws.p2, per, ostride, ooff, tok,
                                        margin);
  }

  void verifier_mfma(const Ws& ws, int B, int C, const T* vision, int vis_ld, int vis_off, T* kv,
                     float* hid, bool head_all, int32_t* tok, int per, int ostride,
                     float* logits, float* margin, int32_t* route_idx, float* route_gap,
                     bool embedded, float* layer_h) {
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim;
    const int L = c.n_layers, E = c.n_routed, k = c.top_k, I = c.moe_inter, S = c.n_shared;
    const int SI = S * I;
    const float eps = (float)c.rms_eps;
    const size_t seq_stride = (size_t)2 * nh * c.max_ctx * dh;
    const size_t layer_stride = (size_t)B * seq_stride;
    const bool small = R <= SR_MAX;  // MoE down adds straight into h
    const unsigned G = groups(R);
    if (!embedded)
      k_embed<BF><<<R, 256, H * sizeof(float), s>>>(R, C, H, c.vocab, ws.row_valid, ws.row_tok,
                                                  (const T*)w.embed, vision, vis_ld, vis_off, ws.h,
                                                  ws.status);
    for (int l = 0; l < L; ++l) {
      const uint16_t* xg = nullptr;
      if (!small) {  // add the previous layer's expert slots (if any), normalise once
        k_combine_norm<<<R, H / 4, 0, s>>>(H, k, l > 0 ? ws.slot : nullptr, ws.h,
                                         w.attn_norm + (size_t)l * H, eps, nullptr,
                                         (uint16_t*)ws.xin);
        xg = (const uint16_t*)ws.xin;
      }
      snap_h(layer_h, l, R);  // after the previous layer's slots were added
      attn_mfma(ws, B, C, w.attn_norm + (size_t)l * H, xg, pk.wqkv + l * pk.wqkv_s,
                pk.wo + l * pk.wo_s, (uint16_t*)kv + (size_t)l * layer_stride, seq_stride);
      if (small && moe_blocks > 0 && ws.moe_sync && ws.lg) {  // router, gate/up, down: one launch
        const unsigned items = (unsigned)((E + 15) / 16 + SI / 16 + E * (I / 16) +
                                          (E + S) * ((H / 16 + 3) / 4));
        const unsigned grid = (unsigned)moe_blocks < items ? (unsigned)moe_blocks : items;
#define MTP_MOE(M)                                                                              \
  launch_k(tm, MTP_KC_MOE, k_s_moe<M>, dim3(grid), dim3(256), lds_rows(R, H), s, R,  \
           H, E, k, I, S, ws.h, w.ffn_norm + (size_t)l * H, eps, pk.router + l * pk.router_s,    \
           w.router_bias ? w.router_bias + (size_t)l * E : nullptr,                              \
           pk.exp_gu + (size_t)l * E * pk.exp_gu_s, pk.exp_gu_s, pk.sh_gu + l * pk.sh_gu_s,      \
           pk.exp_down + (size_t)l * E * pk.exp_down_s, pk.exp_down_s,                           \
           pk.sh_down + l * pk.sh_down_s, ws.lg, (uint16_t*)ws.act, ws.act_sh, ws.dn_part,       \
           ws.moe_sync + (size_t)l * kMoeSyncWords,                                              \
           route_idx ? route_idx + (size_t)l * R * k : nullptr,                                  \
           route_gap ? route_gap + (size_t)l * R : ws.rgap, ws.status, kMoeSpinMax)
        MTP_MAXT_DISPATCH(H / 128, MTP_MOE);
#undef MTP_MOE
        continue;
      }
#define MTP_ROUTER(M)                                                                           \
  launch_k(tm, MTP_KC_ROUTER, k_s_router<M>, dim3(G), dim3(1024), lds_rows(R, H), s, R, H, E, k, \
           ws.h, w.ffn_norm + (size_t)l * H, eps, (uint16_t*)ws.xin, pk.router + l * pk.router_s, \
           w.router_bias ? w.router_bias + (size_t)l * E : nullptr, ws.ridx, ws.rw,               \
           route_gap ? route_gap + (size_t)l * R : ws.rgap,                                       \
           route_idx ? route_idx + (size_t)l * R * k : nullptr, ws.cnt, ws.off, ws.ent_row,       \
           ws.ent_slot, ws.ent_w, ws.touched, ws.n_touched)
      MTP_MAXT_DISPATCH(H / 128, MTP_ROUTER);
#undef MTP_ROUTER
      // more than 16 rows: grouping with 64-entry chunk blocks (the grouped
      // GEMMs' row tile)
      if (G > 1)
        k_group<<<1, 1024, 0, s>>>(R, E, k, ws.ridx, ws.rw, ws.cnt, ws.off, ws.ent_row,
                                   ws.ent_slot, ws.ent_w, kGemmM / 16, ws.cbp);
      const unsigned chunks = (unsigned)(E + cdiv((size_t)R * k, kGemmM)) + cdiv(R, kGemmM);
      if (G == 1) {  // persistent streaming form: two blocks per compute unit
        const uint4* egu = pk.exp_gu + (size_t)l * E * pk.exp_gu_s;
        const uint4* sgu = pk.sh_gu + l * pk.sh_gu_s;
#define MTP_GU(M)                                                                              \
  launch_k(tm, MTP_KC_MOE_GU, k_s_gu_stream<M>, dim3(2 * n_cu), dim3(256), lds_rows(R, H), s, R, \
           H, I, SI, (const uint16_t*)ws.xin, egu, pk.exp_gu_s, sgu, ws.cnt, ws.off, ws.ent_row, \
           ws.touched, ws.n_touched, (uint16_t*)ws.act, ws.act_sh)
        MTP_MAXT_DISPATCH(H / 128, MTP_GU);
#undef MTP_GU
      } else {  // grouped GEMM on the compact grid (blocks past the last item exit)
        const unsigned nblk = grid_xcd((E + cdiv((size_t)R * k, kGemmM)) * (I / kGemmN) +
                                       cdiv(R, kGemmM) * (SI / kGemmN));
        launch_k(tm, MTP_KC_MOE_GU, prefill ? k_gu_gemm<GU_PREFILL> : k_gu_gemm<GU_VERIFY>,
                 dim3(nblk), dim3(256), 0, s, R, H, E, I, SI, (const uint16_t*)ws.xin,
                 pk.exp_gu + (size_t)l * E * pk.exp_gu_s, pk.exp_gu_s,
                 pk.sh_gu + l * pk.sh_gu_s, ws.cnt, ws.off, ws.ent_row, (uint16_t*)ws.act,
                 ws.act_sh, ws.cbp);
      }
      const uint4* edn = pk.exp_down + (size_t)l * E * pk.exp_down_s;
      const uint4* sdn = pk.sh_down + l * pk.sh_down_s;
      if (small) {
        launch_k(tm, MTP_KC_MOE_DOWN, k_s_down_split<kDownSplit>, dim3(H / 16, kDownSplit),
                 dim3(256), 0, s, R, H, E, I, S, (const uint16_t*)ws.act, ws.act_sh, edn,
                 pk.exp_down_s, sdn, ws.cnt, ws.off, ws.ent_row, ws.ent_w, ws.touched,
                 ws.n_touched, ws.dn_part, ws.dn_ctr, ws.h, ws.status);
      } else if (R <= kSlotRows) {  // few entries per expert: 16-entry slot blocks
#define MTP_DSLOT(M)                                                                           \
  launch_k(tm, MTP_KC_MOE_DOWN, k_s_down_slot<M>, dim3(H / 16, E + 1, G), dim3(256), 0, s, 1, R, \
           E, k, H, I, SI, (const uint16_t*)ws.act, ws.act_sh, edn, pk.exp_down_s, sdn, ws.cnt,  \
           ws.off, ws.ent_row, ws.ent_slot, ws.ent_w, ws.slot)
        MTP_MAXT_DISPATCH(I / 128, MTP_DSLOT);
#undef MTP_DSLOT
      } else
        launch_k(tm, MTP_KC_MOE_DOWN, k_down_gemm, dim3(grid_xcd(chunks * (H / kGemmN))), dim3(256), 0, s,
                 R, E, k, H, I, SI, (const uint16_t*)ws.act, ws.act_sh, edn, pk.exp_down_s, sdn,
                 ws.cnt, ws.off, ws.ent_row, ws.ent_slot, ws.ent_w, ws.slot, ws.cbp);
    }
    if (small && tok && head_all) {  // final norm (hid) with the LM head (one launch up to 4 rows)
      snap_h(layer_h, L, R);
      head_norm(ws, R, ws.h, nullptr, w.final_norm, hid, logits, c.vocab, per, ostride, 0, tok,
                margin);
      return;
    }
    uint16_t* xh = (tok && head_all) ? (uint16_t*)ws.xhead : nullptr;
    if (small)
      norm_rows(R, ws.h, nullptr, w.final_norm, hid, xh);
    else  // (adds the last layer's expert slots to h first)
      k_combine_norm<<<R, H / 4, 0, s>>>(H, k, ws.slot, ws.h, w.final_norm, eps, hid, xh);
    snap_h(layer_h, L, R);
    if (!tok) return;
    if (head_all)
      lm_mfma(ws, R, logits, c.vocab, per, ostride, 0, tok, margin);
    else
      head_norm(ws, B, ws.h, ws.head_row, w.final_norm, nullptr, logits, c.vocab, 1, 1, 0, tok,
                margin);
  }

  // Draft-head objective: u = N_o(z) of n rows of ws.h (float32 to u) with
  // the LM-head input in ws.xhead, and LM-head logits of the n rows of
  // ws.xhead ([n][V], row stride V; the argmax goes to ws.tok_stage)
  void obj_final(const Ws& ws, int n, float* u) {
    if constexpr (BF) {
      norm_rows(n, ws.h, nullptr, w.final_norm, u, (uint16_t*)ws.xhead);
    } else {
      k_rmsnorm<BF><<<n, 256, 0, s>>>(c.hidden, ws.h, c.hidden, nullptr, w.final_norm,
                                      (float)c.rms_eps, u, c.hidden, (T*)ws.xhead, c.hidden, 0);
    }
  }
  void obj_logits(const Ws& ws, int n, float* logits) {
    if constexpr (BF) lm_mfma(ws, n, logits, c.vocab, 1, 1, 0, ws.tok_stage, nullptr);
    else lm_head(ws, n, logits, c.vocab, 1, 1, 0, ws.tok_stage, nullptr);
  }

  void draft_mfma(const Ws& ws, int B, int C, const float* a, size_t a_ld, const T* vision,
                  int vis_ld, int vis_off, T* dkv, bool head, int32_t* tok, int ostride, int ooff,
                  float* logits, size_t ldl, bool xin_ready, bool defer_argmax, bool kv_only) {
    const int R = B * C, H = c.hidden, nh = c.n_heads, dh = c.head_dim;
    const int F = c.draft_inter;
    const float eps = (float)c.rms_eps;
    const size_t seq_stride = (size_t)2 * nh * c.max_ctx * dh;
    if (!xin_ready)
      k_draft_in<BF><<<R, 256, 2 * H * sizeof(float), s>>>(
          C, H, c.vocab, ws.row_valid, ws.row_tok, (const T*)w.embed, vision, vis_ld, vis_off, a,
          a_ld, w.d_enorm, w.d_hnorm, eps, (T*)ws.xin, ws.status);
    smm(ws, R, H, 2 * H, (const uint16_t*)ws.xin, 2 * H, pk.d_eh, ws.h, H, false);
    // Up to 16 rows the products normalise their rows in a prologue; with
    // several row groups the rows are normalised once (bf16, into xin) and
    // the products read them, each weight tile applied to cpb groups.
    const unsigned G = groups(R);
    const bool pre = G > 1;
    const uint16_t* xn = pre ? (const uint16_t*)ws.xin : nullptr;
    if (pre) norm_rows(R, ws.h, nullptr, w.d_attn_norm, nullptr, (uint16_t*)ws.xin);
    attn_mfma(ws, B, C, w.d_attn_norm, xn, pk.d_qkv, pk.d_wo, (uint16_t*)dkv, seq_stride,
              kv_only);
    if (kv_only) return;
    if (pre) norm_rows(R, ws.h, nullptr, w.d_ffn_norm, nullptr, (uint16_t*)ws.xin);
    if (pre) {  // tiled GEMM over the normalised rows
      DenseOut o{};
      o.act = ws.act_sh;
      dense<DG_SWIGLU>(ws, MTP_KC_DRAFT_FFN, R, F, H, xn, H, pk.d_gu, o);
    } else {
#define MTP_DFFN(M)                                                                             \
  launch_k(tm, MTP_KC_DRAFT_FFN, prefill ? k_s_gu<GU_DRAFT_PREFILL, M> : k_s_gu<GU_DRAFT, M>,   \
           dim3(F / 16), dim3(256), lds_rows(R, H), s, R, H, F, ws.h, w.d_ffn_norm, eps, pk.d_gu, \
           ws.act_sh)
      MTP_MAXT_DISPATCH(H / 128, MTP_DFFN);
#undef MTP_DFFN
    }
    smm(ws, R, H, F, ws.act_sh, F, pk.d_down, ws.h, H, true);
    if (!head) return;
    head_norm(ws, B, ws.h, ws.head_row, w.final_norm, ws.ustate, logits, ldl, 1, ostride, ooff,
              tok, nullptr, defer_argmax);
  }
};


mtp_status launch_status() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    fprintf(stderr, "mtp: HIP error %s\n", hipGetErrorString(e));
    return MTP_EHIP;
  }
  return MTP_OK;
}

bool ws_ok(const mtp_ctx* ctx, int B, int C, const void* ws, size_t ws_bytes) {
  return ws && carve(ctx->cfg, B, C, nullptr, ctx->n_split).bytes <= ws_bytes;
}

// Repacks every matrix of a bf16 model into MFMA operand tiles (one
// allocation, owned by the context).
mtp_status pack_weights(mtp_ctx* ctx) {
  const mtp_config& c = ctx->cfg;
  const mtp_weights& w = ctx->w;
  const int L = c.n_layers, H = c.hidden, D = c.n_heads * c.head_dim, E = c.n_routed;
  const int I = c.moe_inter, SI = c.n_shared * I, F = c.draft_inter, V = c.vocab;
  Packed& p = ctx->pk;
  p.wqkv_s = packed_elems(3 * D, H);
  p.wo_s = packed_elems(H, D);
  p.router_s = packed_elems(E, H);
  p.exp_gu_s = packed_elems(2 * I, H);
  p.exp_down_s = packed_elems(H, I);
  p.sh_gu_s = packed_elems(2 * SI, H);
  p.sh_down_s = packed_elems(H, SI);
  const size_t lm_s = packed_elems(V, H);
  const size_t eh_s = packed_elems(H, 2 * H), dq_s = packed_elems(3 * D, H);
  const size_t dwo_s = packed_elems(H, D), dgu_s = packed_elems(2 * F, H);
  const size_t ddn_s = packed_elems(H, F);
  const size_t total = L * (p.wqkv_s + p.wo_s + p.router_s + E * (p.exp_gu_s + p.exp_down_s) +
                            p.sh_gu_s + p.sh_down_s) +
                       lm_s + eh_s + dq_s + dwo_s + dgu_s + ddn_s;
  if (hipMalloc(&p.base, total * sizeof(uint4)) != hipSuccess) {
    p.base = nullptr;
    return MTP_EHIP;
  }
  ctx->pk_bytes = total * sizeof(uint4);
  uint4* cur = p.base;
  auto pack = [&](const void* src, size_t src_stride, int count, int N, int K,
                  const uint4** dst) {
    *dst = cur;
    const size_t n = packed_elems(N, K);
    for (int i = 0; i < count; ++i) {
      k_pack<<<cdiv(n, 256), 256>>>((const uint16_t*)src + (size_t)i * src_stride, N, K, cur);
      cur += n;
    }
  };
  pack(w.wqkv, (size_t)3 * D * H, L, 3 * D, H, &p.wqkv);
  pack(w.wo, (size_t)H * D, L, H, D, &p.wo);
  pack(w.router, (size_t)E * H, L, E, H, &p.router);
  pack(w.exp_gu, (size_t)2 * I * H, L * E, 2 * I, H, &p.exp_gu);
  pack(w.exp_down, (size_t)H * I, L * E, H, I, &p.exp_down);
  pack(w.sh_gu, (size_t)2 * SI * H, L, 2 * SI, H, &p.sh_gu);
  pack(w.sh_down, (size_t)H * SI, L, H, SI, &p.sh_down);
  pack(c.tie_lm_head ? w.embed : w.lm_head, 0, 1, V, H, &p.lm);
  pack(w.d_eh_proj, 0, 1, H, 2 * H, &p.d_eh);
  pack(w.d_wqkv, 0, 1, 3 * D, H, &p.d_qkv);
  pack(w.d_wo, 0, 1, H, D, &p.d_wo);
  pack(w.d_gu, 0, 1, 2 * F, H, &p.d_gu);
  pack(w.d_down, 0, 1, H, F, &p.d_down);
  if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) return MTP_EHIP;
  return MTP_OK;
}

}  // namespace

extern "C" {

mtp_status mtp_create(const mtp_config* cfg, const mtp_weights* w, mtp_ctx** out) {
  if (!cfg || !w || !out) return MTP_EINVAL;
  *out = nullptr;
  const mtp_config& c = *cfg;
  if (c.n_layers < 1 || c.hidden < 64 || c.n_heads < 1 || c.n_routed < 1 || c.top_k < 1 ||
      c.top_k > c.n_routed || c.n_shared < 1 || c.moe_inter < 4 || c.draft_inter < 4 ||
      c.vocab < 2 || c.max_batch < 1 || c.max_ctx < 2 || c.max_k < 0 || c.rope_theta <= 0 ||
      c.rms_eps < 0 || (c.dtype != MTP_F32 && c.dtype != MTP_BF16))
    return MTP_EINVAL;
  if (c.hidden % 64 || (c.head_dim != 64 && c.head_dim != 128) || c.n_routed > 64 ||
      c.moe_inter % 4 || c.draft_inter % 4 || (c.n_heads * c.head_dim) % 64)
    return MTP_EUNSUPPORTED;
  // bf16 MFMA path: contraction lengths multiples of 128, whole float4 rows
  // per lane (hidden % 256, <= 2048), top-k <= 8
  if (c.dtype == MTP_BF16 && (c.hidden % 256 || c.hidden > 2048 ||
                              (c.n_heads * c.head_dim) % 128 || c.moe_inter % 128 ||
                              c.draft_inter % 128 || c.top_k > 8))
    return MTP_EUNSUPPORTED;
  if (!w->embed || (!c.tie_lm_head && !w->lm_head) || !w->final_norm || !w->attn_norm ||
      !w->ffn_norm || !w->wqkv || !w->wo || !w->router || !w->exp_gu || !w->exp_down ||
      !w->sh_gu || !w->sh_down || !w->d_enorm || !w->d_hnorm || !w->d_attn_norm ||
      !w->d_ffn_norm || !w->d_eh_proj || !w->d_wqkv || !w->d_wo || !w->d_gu || !w->d_down)
    return MTP_EINVAL;
  mtp_ctx* ctx = new (std::nothrow) mtp_ctx;
  if (!ctx) return MTP_EINVAL;
  ctx->cfg = c;
  ctx->w = *w;
  ctx->rope = nullptr;
  ctx->dstatus = nullptr;
  ctx->scratch = nullptr;
  ctx->pk = Packed{};
  ctx->pk_bytes = 0;
  {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, dev) !=
            hipSuccess ||
        ctx->n_cu < 1) {
      delete ctx;
      return MTP_EHIP;
    }
  }
  // key splits for decode attention: about 128 positions each, at most 64
  ctx->n_split = (c.max_ctx + 127) / 128;
  if (ctx->n_split > 64) ctx->n_split = 64;
  ctx->spl = ((c.max_ctx + ctx->n_split - 1) / ctx->n_split + 63) / 64 * 64;
  ctx->n_split = (c.max_ctx + ctx->spl - 1) / ctx->spl;
  const int half = c.head_dim / 2;
  const size_t n = (size_t)c.max_ctx * half;
  float2* host = new (std::nothrow) float2[n];
  if (!host) {
    delete ctx;
    return MTP_EINVAL;
  }
  for (int p = 0; p < c.max_ctx; ++p)
    for (int i = 0; i < half; ++i) {
      double inv = std::pow(c.rope_theta, -2.0 * i / c.head_dim);
      double ang = (double)p * inv;
      host[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
    }
  if (hipMalloc(&ctx->rope, n * sizeof(float2)) != hipSuccess ||
      hipMemcpy(ctx->rope, host, n * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess) {
    delete[] host;
    if (ctx->rope) (void)hipFree(ctx->rope);
    delete ctx;
    return MTP_EHIP;
  }
  delete[] host;
  if (hipMalloc(&ctx->dstatus, 256) != hipSuccess ||
      hipMemset(ctx->dstatus, 0, 256) != hipSuccess || scratch_addr(&ctx->scratch) != MTP_OK) {
    mtp_destroy(ctx);
    return MTP_EHIP;
  }
  ctx->moe_blocks = 0;
  if (c.dtype == MTP_BF16) {
    mtp_status st = pack_weights(ctx);
    if (st != MTP_OK) {
      mtp_destroy(ctx);
      return st;
    }
    ctx->moe_blocks = moe_resident_blocks(c, ctx->n_cu);
  }
  *out = ctx;
  return MTP_OK;
}

static void timing_release(Timing& t) {
  if (t.ev) {
    for (int i = 0; i < 2 * t.cap; ++i)
      if (t.ev[i]) (void)hipEventDestroy(t.ev[i]);
    delete[] t.ev;
  }
  t = Timing{};
}

void mtp_destroy(mtp_ctx* ctx) {
  if (!ctx) return;
  timing_release(ctx->tm);
  if (ctx->rope) (void)hipFree(ctx->rope);
  if (ctx->dstatus) (void)hipFree(ctx->dstatus);
  if (ctx->pk.base) (void)hipFree(ctx->pk.base);
  delete ctx;
}

size_t mtp_context_bytes(const mtp_ctx* ctx) {
  if (!ctx) return 0;
  return (size_t)ctx->cfg.max_ctx * (ctx->cfg.head_dim / 2) * sizeof(float2) + 256 +
         ctx->pk_bytes;
}

size_t mtp_workspace_bytes(const mtp_ctx* ctx, int32_t batch, int32_t rows) {
  if (!ctx || batch < 1 || rows < 1) return 0;
  return carve(ctx->cfg, batch, rows, nullptr, ctx->n_split).bytes;
}

mtp_status mtp_status_read(const mtp_ctx* ctx, const void* ws, int32_t* status) {
  if (!ctx || !status) return MTP_EINVAL;
  int32_t w = 0, c = 0;
  if (ws && hipMemcpy(&w, ws, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess)
    return MTP_EHIP;
  if (hipMemcpy(&c, ctx->dstatus, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess)
    return MTP_EHIP;
  *status = w != 0 ? w : c;
  return MTP_OK;
}

mtp_status mtp_status_clear(const mtp_ctx* ctx, void* ws, void* stream) {
  if (!ctx) return MTP_EINVAL;
  if (ws) k_fill_i32<<<1, 64, 0, (hipStream_t)stream>>>((int32_t*)ws, 1, 0);
  k_fill_i32<<<1, 64, 0, (hipStream_t)stream>>>(ctx->dstatus, 1, 0);
  return launch_status();
}

mtp_status mtp_prefill(mtp_ctx* ctx, int32_t batch, int32_t k, int32_t n_rows, const int32_t* tok,
                       const void* vision, void* kv_cache, void* draft_kv, int32_t* kv_len,
                       int32_t* draft_len, float* hid, int32_t* next_tok, int32_t* n_rows_out,
                       int32_t* row_pos, int32_t* pending, int32_t* out_tok, int32_t max_out,
                       int32_t* n_out, int32_t* route_idx, void* ws, size_t ws_bytes,
                       void* stream) {
  if (!ctx) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || k < 0 || k > c.max_k || n_rows < 1 ||
      n_rows > c.max_ctx || !tok || !kv_cache || !draft_kv || !kv_len || !draft_len || !hid ||
      !next_tok || !n_rows_out || !row_pos || !pending || !n_out || max_out < 0 ||
      (max_out > 0 && !out_tok) || !ws)
    return MTP_EINVAL;
  // largest chunk whose workspace fits
  int C = 0;
  for (int t = n_rows; t >= 1; t = t > 64 ? t / 2 : t - 1)
    if (carve(c, batch, t, nullptr, ctx->n_split).bytes <= ws_bytes) {
      C = t;
      break;
    }
  if (C < 1) return MTP_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  auto run = [&](auto tag) -> mtp_status {
    constexpr bool BF = decltype(tag)::value;
    using T = typename St<BF>::T;
    Model<BF> m{c, ctx->w, ctx->rope, s, ctx->pk, ctx->n_split, ctx->spl, &ctx->tm, ctx->n_cu, ctx->moe_blocks};
    m.prefill = true;
    Ws w = carve(c, batch, C, ws, ctx->n_split);
    for (int c0 = 0; c0 < n_rows; c0 += C) {
      const int Cc = n_rows - c0 < C ? n_rows - c0 : C;
      const int R = batch * Cc;
      const bool last = c0 + Cc == n_rows;
      k_rows_setup<<<cdiv(R, 256), 256, 0, s>>>(batch, Cc, nullptr, c0, nullptr, c.max_ctx,
                                                 w.row_pos, w.row_valid, w.head_row, w.status,
                                                 w.att_ctr, w.n_ctr);
      k_row_tokens<<<cdiv(R, 256), 256, 0, s>>>(batch, Cc, tok, n_rows, c0, w.row_tok);
      m.pos_end = c0 + Cc;  // this pass's rows and the draft prefill's sit at c0..c0+Cc-1
      m.verifier(w, batch, Cc, (const T*)vision, n_rows, c0, (T*)kv_cache, w.bbuf, false,
                 last ? w.tok_stage : nullptr, 1, 1, nullptr, nullptr,
                 route_idx ? w.route_stage : nullptr, nullptr);
      if (route_idx) {
        const size_t n = (size_t)c.n_layers * R * c.top_k;
        k_scatter_routes<<<cdiv(n, 256) < 1024 ? cdiv(n, 256) : 1024, 256, 0, s>>>(
            c.n_layers, batch, Cc, c.top_k, n_rows, c0, w.route_stage, route_idx);
      }
      if (last)
        k_copy_rows<<<batch, 256, 0, s>>>(batch, c.hidden, w.head_row, w.bbuf, hid,
                                          (size_t)(k + 1) * c.hidden);
      // draft prefill: rows p = c0..c0+Cc-1 with p <= n_rows-2, input row p+1
      const int nv = (n_rows - 1 - c0) < Cc ? (n_rows - 1 - c0) : Cc;
      if (nv > 0) {
        k_fill_i32<<<cdiv(batch, 256), 256, 0, s>>>(w.chain_pos, batch, nv);
        k_rows_setup<<<cdiv(R, 256), 256, 0, s>>>(batch, Cc, nullptr, c0, w.chain_pos, c.max_ctx,
                                                   w.row_pos, w.row_valid, nullptr, w.status);
        k_row_tokens<<<cdiv(R, 256), 256, 0, s>>>(batch, Cc, tok, n_rows, c0 + 1, w.row_tok);
        m.draft(w, batch, Cc, w.bbuf, (size_t)Cc * c.hidden, (const T*)vision, n_rows, c0 + 1,
                (T*)draft_kv, false, nullptr, 0, 0, nullptr, 0, false, false, /*kv_only=*/true);
      }
    }
    k_prefill_state<<<cdiv(batch, 256), 256, 0, s>>>(batch, k, n_rows, w.tok_stage, kv_len,
                                                     draft_len, next_tok, n_rows_out, row_pos,
                                                     pending, out_tok, max_out, n_out);
    return launch_status();
  };
  if (c.dtype == MTP_BF16) return run(std::true_type{});
  return run(std::false_type{});
}

mtp_status mtp_draft_k(mtp_ctx* ctx, int32_t batch, int32_t k, const float* hid,
                       const int32_t* next_tok, const int32_t* n_rows, const int32_t* row_pos,
                       void* draft_kv, int32_t* draft_len, int32_t* draft_tok,
                       float* draft_logits, float* draft_u, void* ws, size_t ws_bytes,
                       void* stream) {
  if (!ctx) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || k < 0 || k > c.max_k) return MTP_EINVAL;
  if (k == 0) return MTP_OK;
  if (!hid || !next_tok || !n_rows || !row_pos || !draft_kv || !draft_len || !draft_tok ||
      !ws_ok(ctx, batch, k + 1, ws, ws_bytes))
    return MTP_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  auto run = [&](auto tag) -> mtp_status {
    constexpr bool BF = decltype(tag)::value;
    using T = typename St<BF>::T;
    Model<BF> m{c, ctx->w, ctx->rope, s, ctx->pk, ctx->n_split, ctx->spl, &ctx->tm, ctx->n_cu, ctx->moe_blocks};
    const int C = k + 1, R = batch * C, H = c.hidden, V = c.vocab;
    Ws w = carve(c, batch, C, ws, ctx->n_split);
    const float eps = (float)c.rms_eps;
    const int n4 = H / 256;  // float4 per lane of a row (bf16 model)
    // the draft block's counters (attention, down strips): the fused MoE's
    // words after them belong to verify passes, whose first kernel clears them
    const int n_zero = (int)(w.moe_sync ? w.moe_sync - w.att_ctr : w.n_ctr);
    // depth 1 over the catch-up rows; the last valid row starts the chain
    if constexpr (BF) {
#define MTP_DRI(NV)                                                                          \
  k_draft_rows_in<NV><<<R, 64, 0, s>>>(batch, C, row_pos, n_rows, next_tok, c.max_ctx, H, V, \
                                       (const uint16_t*)ctx->w.embed, hid, (size_t)C * H,     \
                                       ctx->w.d_enorm, ctx->w.d_hnorm, eps, w.row_pos,        \
                                       w.row_valid, w.head_row, w.row_tok, draft_len, w.status, \
                                       w.att_ctr, n_zero, (uint16_t*)w.xin)
      MTP_NV_DISPATCH(n4, MTP_DRI);
#undef MTP_DRI
    } else {
      k_draft_rows<<<cdiv(R, 256), 256, 0, s>>>(batch, C, row_pos, n_rows, next_tok, c.max_ctx,
                                                 w.row_pos, w.row_valid, w.head_row, w.row_tok,
                                                 draft_len, w.status, w.att_ctr, n_zero);
    }
    // depth d's output state u (ws.ustate, [B][H]) into draft_u[b][d-1]
    auto keep_u = [&](int d) {
      if (draft_u)
        (void)hipMemcpy2DAsync(draft_u + (size_t)(d - 1) * H, (size_t)k * H * sizeof(float),
                               w.ustate, (size_t)H * sizeof(float), (size_t)H * sizeof(float),
                               batch, hipMemcpyDeviceToDevice, s);
    };
    m.draft(w, batch, C, hid, (size_t)C * H, nullptr, 0, 0, (T*)draft_kv, true, draft_tok, k, 0,
            draft_logits, (size_t)k * V, BF, BF && k > 1);
    keep_u(1);
    const unsigned nbp = m.lm_partials(batch);
    // depth d = 2..k: one row at (row_pos + n_rows - 1) + (d - 1), state u
    // of depth d-1 (read by the draft input before the head rewrites it),
    // input the depth d-1 draft token
    for (int d = 2; d <= k; ++d) {
      if constexpr (BF) {
#define MTP_CRI(NV)                                                                           \
  k_chain_rows_in<NV><<<batch, 256, 0, s>>>(batch, d, k, row_pos, n_rows, (int)nbp, w.pv, w.pi, \
                                            w.p2, draft_tok, c.max_ctx, H, V,                  \
                                            (const uint16_t*)ctx->w.embed, w.ustate,           \
                                            ctx->w.d_enorm, ctx->w.d_hnorm, eps, w.row_pos,    \
                                            w.row_valid, w.head_row, w.row_tok, w.status,      \
                                            (uint16_t*)w.xin)
        MTP_NV_DISPATCH(n4, MTP_CRI);
#undef MTP_CRI
      } else {
        k_chain_rows<<<cdiv(batch, 256), 256, 0, s>>>(batch, d, k, row_pos, n_rows, draft_tok,
                                                       c.max_ctx, w.row_pos, w.row_valid,
                                                       w.head_row, w.row_tok, w.status);
      }
      m.draft(w, batch, 1, w.ustate, (size_t)H, nullptr, 0, 0, (T*)draft_kv, true, draft_tok, k,
              d - 1, draft_logits ? draft_logits + (size_t)(d - 1) * V : nullptr, (size_t)k * V,
              BF, BF && d < k);
      keep_u(d);
    }
    return launch_status();
  };
  if (c.dtype == MTP_BF16) return run(std::true_type{});
  return run(std::false_type{});
}

mtp_status moe_verify_step(mtp_ctx* ctx, int32_t batch, int32_t k, const int32_t* pending,
                           const int32_t* draft_tok, const int32_t* kv_len, void* kv_cache,
                           int32_t* verify_tok, float* hid, float* logits, float* margin,
                           int32_t* route_idx, float* route_gap, float* layer_h, void* ws,
                           size_t ws_bytes, void* stream) {
  if (!ctx) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || k < 0 || k > c.max_k || !pending ||
      (k > 0 && !draft_tok) || !kv_len || !kv_cache || !verify_tok || !hid ||
      !ws_ok(ctx, batch, k + 1, ws, ws_bytes))
    return MTP_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  auto run = [&](auto tag) -> mtp_status {
    constexpr bool BF = decltype(tag)::value;
    using T = typename St<BF>::T;
    Model<BF> m{c, ctx->w, ctx->rope, s, ctx->pk, ctx->n_split, ctx->spl, &ctx->tm, ctx->n_cu, ctx->moe_blocks};
    const int C = k + 1, R = batch * C;
    Ws w = carve(c, batch, C, ws, ctx->n_split);
    k_verify_rows<BF><<<verify_rows_grid(R, w.n_ctr), 256, 0, s>>>(
        batch, k, kv_len, pending, draft_tok, c.max_ctx, c.hidden, c.vocab,
        (const T*)ctx->w.embed, w.row_pos, w.row_valid, w.h, w.status, w.att_ctr, w.n_ctr);
    m.verifier(w, batch, C, nullptr, 0, 0, (T*)kv_cache, hid, true, verify_tok, R, 0, logits,
               margin, route_idx, route_gap, /*embedded=*/true, layer_h);
    return launch_status();
  };
  if (c.dtype == MTP_BF16) return run(std::true_type{});
  return run(std::false_type{});
}

mtp_status moe_verify_step_static(mtp_ctx* ctx, int32_t batch, int32_t k,
                                  const int32_t* pending, const int32_t* draft_tok,
                                  const int32_t* kv_len, void* kv_cache, int32_t* verify_tok,
                                  float* hid, float* logits, float* margin, int32_t* route_idx,
                                  float* route_gap, float* layer_h, void* stream) {
  if (!ctx || !ctx->scratch) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || k < 0 || k > c.max_k || !pending ||
      (k > 0 && !draft_tok) || !kv_len || !kv_cache || !verify_tok || !hid)
    return MTP_EINVAL;
  if (carve(c, batch, k + 1, nullptr, ctx->n_split).bytes > kScratchBytes) {
    fprintf(stderr,
            "moe_verify_step_static: %d sequences x %d rows need %zu scratch bytes, more than "
            "the %zu of the static scratch\n",
            batch, k + 1, carve(c, batch, k + 1, nullptr, ctx->n_split).bytes, kScratchBytes);
    return MTP_EUNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  auto run = [&](auto tag) -> mtp_status {
    constexpr bool BF = decltype(tag)::value;
    using T = typename St<BF>::T;
    Model<BF> m{c, ctx->w, ctx->rope, s, ctx->pk, ctx->n_split, ctx->spl, &ctx->tm, ctx->n_cu, ctx->moe_blocks};
    const int C = k + 1, R = batch * C;
    Ws w = carve(c, batch, C, ctx->scratch, ctx->n_split);
    w.status = ctx->dstatus;  // device conditions go to the context's status word
    k_verify_rows<BF><<<verify_rows_grid(R, w.n_ctr), 256, 0, s>>>(
        batch, k, kv_len, pending, draft_tok, c.max_ctx, c.hidden, c.vocab,
        (const T*)ctx->w.embed, w.row_pos, w.row_valid, w.h, w.status, w.att_ctr, w.n_ctr);
    m.verifier(w, batch, C, nullptr, 0, 0, (T*)kv_cache, hid, true, verify_tok, R, 0, logits,
               margin, route_idx, route_gap, /*embedded=*/true, layer_h);
    return launch_status();
  };
  if (c.dtype == MTP_BF16) return run(std::true_type{});
  return run(std::false_type{});
}

// ---------------------------------------------------------------- objective
constexpr int kObjMaxK = 8;     // depths of the objective
// draft rows per pass: a pass reads the LM head's weights (331 MB at the
// full shape) four times, so the fewer passes the better (measured at 1,279
// draft rows: passes of 256 rows 559,013 grid rows/s, of 512 662,776, one
// pass 830,477); a pass's logits take 2 * rows * V * 4 bytes of workspace
constexpr int kObjChunk = 1280;

struct ObjWs {
  Ws w;                           // the draft pass over up to kObjChunk rows
  float *a, *u, *lp, *lq, *terms;
  size_t bytes;
};

// u: every depth's outputs [kObjMaxK][n_rows][H] (a depth's rows shift into
// the next depth's states across chunk boundaries)
ObjWs obj_carve(const mtp_config& c, int n_rows, void* base, int n_split) {
  const int C = n_rows - 1 < kObjChunk ? n_rows - 1 : kObjChunk;
  ObjWs o{};
  o.w = carve(c, 1, C, base, n_split);
  size_t off = align_up(o.w.bytes);
  char* p = (char*)base;
  auto take = [&](size_t bytes) {
    float* r = p ? (float*)(p + off) : nullptr;
    off += align_up(bytes);
    return r;
  };
  const size_t H = c.hidden, V = c.vocab;
  o.a = take((size_t)C * H * 4);
  o.u = take((size_t)kObjMaxK * n_rows * H * 4);
  o.lp = take((size_t)C * V * 4);
  o.lq = take((size_t)C * V * 4);
  o.terms = take((size_t)kObjMaxK * n_rows * 3 * 4);
  o.bytes = off;
  return o;
}

size_t mtp_objective_workspace_bytes(const mtp_ctx* ctx, int32_t n_rows) {
  if (!ctx || n_rows < 4 || n_rows > ctx->cfg.max_ctx) return 0;
  return obj_carve(ctx->cfg, n_rows, nullptr, ctx->n_split).bytes;
}

mtp_status mtp_objective(mtp_ctx* ctx, int32_t n_rows, int32_t n_prompt, int32_t k,
                         const int32_t* tok, const void* vision, const float* b_states,
                         void* draft_kv, float* row_terms, float* u_out, double* loss, void* ws,
                         size_t ws_bytes, void* stream) {
  if (!ctx) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (n_rows < 4 || n_rows > c.max_ctx || n_prompt < 1 || n_prompt > n_rows - 3 || k < 1 ||
      k > kObjMaxK || !tok || !b_states || !draft_kv || !loss || !ws ||
      obj_carve(c, n_rows, nullptr, ctx->n_split).bytes > ws_bytes)
    return MTP_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  auto run = [&](auto tag) -> mtp_status {
    constexpr bool BF = decltype(tag)::value;
    using T = typename St<BF>::T;
    Model<BF> m{c, ctx->w, ctx->rope, s, ctx->pk, ctx->n_split, ctx->spl, &ctx->tm, ctx->n_cu,
                ctx->moe_blocks};
    m.prefill = true;
    ObjWs o = obj_carve(c, n_rows, ws, ctx->n_split);
    Ws& w = o.w;
    const int H = c.hidden, V = c.vocab, C = n_rows - 1 < kObjChunk ? n_rows - 1 : kObjChunk;
    const size_t cache = (size_t)2 * c.n_heads * c.max_ctx * c.head_dim;  // one depth's cache
    k_fill_i32<<<1, 64, 0, s>>>(w.status, 1, 0);
    k_fill_i32<<<cdiv((size_t)kObjMaxK * n_rows * 3, 256), 256, 0, s>>>(
        (int32_t*)o.terms, kObjMaxK * n_rows * 3, 0);  // (+0.f)
    // chunks of rows in order; inside a chunk the depths in order, each
    // with its own draft cache, so the verifier logits Q of the chunk's
    // rows are computed once for every depth
    for (int c0 = 0; c0 < n_rows - 1; c0 += C) {
      const int Cc = n_rows - 1 - c0 < C ? n_rows - 1 - c0 : C;
      k_obj_rows_in<BF><<<Cc, 256, 0, s>>>(H, b_states + (size_t)(c0 + 1) * H, (T*)w.xhead);
      m.obj_logits(w, Cc, o.lq);
      m.pos_end = c0 + Cc;  // the draft rows of this chunk sit at c0..c0+Cc-1
      for (int d = 1; d <= k; ++d) {
        float* u_d = o.u + (size_t)(d - 1) * n_rows * H;
        k_fill_i32<<<1, 64, 0, s>>>(w.chain_pos, 1, Cc);
        k_rows_setup<<<cdiv(Cc, 256), 256, 0, s>>>(1, Cc, nullptr, c0, w.chain_pos, c.max_ctx,
                                                    w.row_pos, w.row_valid, w.head_row, w.status,
                                                    w.att_ctr, w.n_ctr);
        k_row_tokens<<<cdiv(Cc, 256), 256, 0, s>>>(1, Cc, tok, n_rows, c0 + 1, w.row_tok);
        k_obj_states<<<Cc, 256, 0, s>>>(c0, H, d, n_prompt, b_states,
                                        d > 1 ? u_d - (size_t)n_rows * H : nullptr, o.a);
        m.draft(w, 1, Cc, o.a, (size_t)H, (const T*)vision, n_rows, c0 + 1,
                (T*)draft_kv + (size_t)(d - 1) * cache, false, nullptr, 0, 0, nullptr, 0);
        m.obj_final(w, Cc, u_d + (size_t)c0 * H);
        m.obj_logits(w, Cc, o.lp);
        k_obj_terms<<<Cc, 256, 0, s>>>(c0, n_rows, n_prompt, V, H, o.lp, o.lq, u_d, b_states,
                                       tok, o.terms + (size_t)(d - 1) * n_rows * 3, w.status);
      }
    }
    k_obj_loss<<<1, 256, 0, s>>>(k, n_rows, n_prompt, 0.6, o.terms, loss);
    if (row_terms)
      (void)hipMemcpyAsync(row_terms, o.terms, (size_t)k * n_rows * 3 * 4,
                           hipMemcpyDeviceToDevice, s);
    if (u_out)
      for (int d = 0; d < k; ++d) {
        float* dst = u_out + (size_t)d * n_rows * H;
        (void)hipMemcpyAsync(dst, o.u + (size_t)d * n_rows * H, (size_t)(n_rows - 1) * H * 4,
                             hipMemcpyDeviceToDevice, s);
        k_fill_i32<<<cdiv(H, 256), 256, 0, s>>>((int32_t*)(dst + (size_t)(n_rows - 1) * H), H,
                                               0);  // (+0.f; no memset node under capture)
      }
    return launch_status();
  };
  if (c.dtype == MTP_BF16) return run(std::true_type{});
  return run(std::false_type{});
}

mtp_status greedy_accept(int32_t batch, int32_t k, const int32_t* draft_tok,
                         const int32_t* verify_tok, int32_t* accept_len, int32_t* commit_tok,
                         void* stream) {
  if (batch < 1 || k < 0 || (k > 0 && !draft_tok) || !verify_tok || !accept_len || !commit_tok)
    return MTP_EINVAL;
  k_accept<<<cdiv(batch, 256), 256, 0, (hipStream_t)stream>>>(batch, k, draft_tok, verify_tok,
                                                               accept_len, commit_tok);
  return launch_status();
}

mtp_status kv_commit_rollback(mtp_ctx* ctx, int32_t batch, int32_t k, const int32_t* accept_len,
                              const int32_t* commit_tok, int32_t* kv_len, int32_t* n_rows,
                              int32_t* row_pos, int32_t* pending, int32_t* next_tok,
                              const int32_t* max_new, int32_t* out_tok, int32_t max_out,
                              int32_t* n_out, void* stream) {
  if (!ctx) return MTP_EINVAL;
  const mtp_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || k < 0 || k > c.max_k || !accept_len || !commit_tok ||
      !kv_len || !n_rows || !row_pos || !pending || !next_tok || max_out < 0 ||
      (max_out > 0 && !out_tok) || !n_out)
    return MTP_EINVAL;
  k_commit<<<cdiv(batch, 256), 256, 0, (hipStream_t)stream>>>(
      batch, k, accept_len, commit_tok, kv_len, n_rows, row_pos, pending, next_tok, max_new,
      out_tok, max_out, n_out, ctx->dstatus);
  return launch_status();
}

mtp_status mtp_bench_override_drafts(int32_t batch, int32_t k, const int32_t* table,
                                     int32_t n_steps, int32_t* step_ctr, int32_t* draft_tok,
                                     void* stream) {
  if (batch < 1 || k < 1 || !table || n_steps < 1 || !step_ctr || !draft_tok) return MTP_EINVAL;
  k_override<<<1, 256, 0, (hipStream_t)stream>>>(batch, k, table, n_steps, step_ctr, draft_tok);
  return launch_status();
}

mtp_status mtp_timing_start(mtp_ctx* ctx, int32_t kernel_class, int32_t max_launches) {
  if (!ctx || kernel_class < MTP_KC_ATTN || kernel_class > MTP_KC_MOE || max_launches < 1 ||
      ctx->tm.kclass != 0)
    return MTP_EINVAL;
  Timing t;
  t.ev = new (std::nothrow) hipEvent_t[2 * (size_t)max_launches]();
  if (!t.ev) return MTP_EHIP;
  t.cap = max_launches;
  for (int i = 0; i < 2 * max_launches; ++i)
    if (hipEventCreateWithFlags(&t.ev[i], hipEventDisableSystemFence) != hipSuccess) {
      timing_release(t);
      return MTP_EHIP;
    }
  t.kclass = kernel_class;
  ctx->tm = t;
  return MTP_OK;
}

mtp_status mtp_timing_stop(mtp_ctx* ctx, float* total_ms, int32_t* n_launches) {
  if (!ctx || ctx->tm.kclass == 0 || !total_ms || !n_launches) return MTP_EINVAL;
  Timing& t = ctx->tm;
  mtp_status st = MTP_OK;
  double sum = 0.0;
  if (t.n > 0 && hipEventSynchronize(t.ev[2 * t.n - 1]) != hipSuccess) st = MTP_EHIP;
  for (int i = 0; i < t.n && st == MTP_OK; ++i) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]) != hipSuccess) st = MTP_EHIP;
    sum += ms;
  }
  *total_ms = (float)sum;
  *n_launches = t.n;
  timing_release(t);
  return st;
}

}  // extern "C"
