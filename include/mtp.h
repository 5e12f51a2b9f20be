/*
 * mtp.h -- C ABI of the MI355X FastMTP greedy speculative-decode step.
 *
 * One decode step of Jina-OCR-v1 (arxiv 2609.03181) is
 *   mtp_draft_k        K draft tokens from one shared FastMTP block applied
 *                      recursively (Section "Draft-head architecture",
 *                      state-shift equation);
 *   moe_verify_step    one verifier pass over the K+1 rows [pending token,
 *                      drafts] -- decode attention over the KV cache, top-k
 *                      routed + shared-expert MoE FFN, final norm, LM head
 *                      and greedy argmax (Table "Model specification");
 *   greedy_accept      the longest equality prefix m of drafts vs verifier
 *                      tokens and the committed tokens x_1..x_m, v_{m+1}
 *                      (acceptance equation and the paragraph after it);
 *   kv_commit_rollback the committed-token cache update: the K/V rows of
 *                      the m+1 committed rows already sit at their absolute
 *                      positions, so commit is a length update and rollback
 *                      discards nothing but the length (no data moves).
 * With k = 0 the same calls are plain greedy decoding.
 *
 * Conventions
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns
 *     and allocates every buffer; step calls never allocate, never copy
 *     to or from the host and never synchronise, so a whole step can be
 *     captured into one HIP graph.  `stream` is a hipStream_t.
 *   - Matrices are row-major [out][in].  Storage dtype (MTP_F32 or
 *     MTP_BF16) applies to weights, embeddings, vision rows and KV caches;
 *     norm gains and router bias are always float32; hidden states and
 *     logits are float32.
 *   - Each call validates its host-side scalars and pointers; a failure
 *     returns MTP_EINVAL and enqueues nothing.  Conditions only visible on
 *     the device (a position past max_ctx, a token id outside the
 *     vocabulary) set a sticky status word in the workspace, read with
 *     mtp_status_read after the caller synchronises; the affected rows are
 *     skipped rather than written out of bounds.  A failed launch returns
 *     MTP_EHIP.  No exception crosses the ABI.
 *   - The workspace `ws` (size mtp_workspace_bytes) must be zero-filled
 *     once before its first use; it holds scratch, self-resetting counters
 *     and the status word.  Calls sharing one workspace must be ordered on
 *     one stream.
 */
#ifndef MTP_H
#define MTP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MTP_OK = 0,
  MTP_EINVAL = -1,       /* bad host argument; nothing enqueued */
  MTP_ECAPACITY = -2,    /* device: a position would pass max_ctx */
  MTP_EHIP = -3,         /* a HIP call failed */
  MTP_EUNSUPPORTED = -4, /* shape outside what the kernels support */
  MTP_ETOKEN = -5,       /* device: a token id outside [0, vocab) */
  MTP_ERANGE = -6,       /* device: a value outside its range (an acceptance length
                            outside [0, k]; a MoE contribution past the fixed-point
                            range of the small-batch down projection) */
  MTP_ESTALL = -7        /* device: a bounded wait between the blocks of a persistent
                            kernel expired (an internal error: the call's outputs are
                            invalid) */
} mtp_status;

enum { MTP_F32 = 0, MTP_BF16 = 1 };

/* (host) model shape and limits. */
typedef struct {
  int32_t n_layers, hidden, n_heads, head_dim;
  int32_t n_routed, top_k, n_shared, moe_inter; /* MoE: E routed, top-k, S shared, width I */
  int32_t draft_inter;                          /* draft dense FFN width F */
  int32_t vocab, tie_lm_head, dtype;            /* dtype: MTP_F32 or MTP_BF16 */
  int32_t max_batch, max_ctx, max_k;            /* limits of every later call */
  double rope_theta, rms_eps;
} mtp_config;

/* (host struct of device pointers) weights; the context keeps the
 * pointers, not copies.  Shapes with L layers, H hidden, D = heads*dim:
 *   embed [V][H]; lm_head [V][H] (ignored when tied); final_norm [H] f32
 *   attn_norm, ffn_norm [L][H] f32; wqkv [L][3D][H] (q rows, k rows, v
 *   rows); wo [L][H][D]; router [L][E][H]; router_bias [L][E] f32 or NULL
 *   exp_gu [L][E][2I][H] (gate rows then up rows); exp_down [L][E][H][I]
 *   sh_gu [L][2SI][H] (gate rows of the S shared experts, then up rows);
 *   sh_down [L][H][SI]
 *   draft: d_enorm, d_hnorm, d_attn_norm, d_ffn_norm [H] f32;
 *   d_eh_proj [H][2H] (embedding half first); d_wqkv [3D][H]; d_wo [H][D];
 *   d_gu [2F][H] (gate rows then up rows); d_down [H][F]. */
typedef struct {
  const void *embed, *lm_head;
  const float* final_norm;
  const float *attn_norm, *ffn_norm;
  const void *wqkv, *wo, *router;
  const float* router_bias;
  const void *exp_gu, *exp_down, *sh_gu, *sh_down;
  const float *d_enorm, *d_hnorm, *d_attn_norm, *d_ffn_norm;
  const void *d_eh_proj, *d_wqkv, *d_wo, *d_gu, *d_down;
} mtp_weights;

typedef struct mtp_ctx mtp_ctx;

/* Cache layouts (storage dtype), with cap = max_ctx:
 *   verifier KV  [L][B][2][nh][cap][dh]   (k then v)
 *   draft KV     [B][2][nh][cap][dh]
 * Position p of sequence b holds the K/V of the row at absolute position p. */

/* Creates a context: validates the shape and makes the library's only
 * device allocations, all owned by the context until mtp_destroy:
 *   - a float32 RoPE table [max_ctx][dh/2] (cos, sin from float64 angles);
 *   - bf16 models: a second copy of every weight matrix except the
 *     embedding table, repacked into the MFMA operand-tile layout the
 *     kernels stream (the embedding table, the norm gains and the router
 *     bias are read in place, so the caller keeps every weight alive until
 *     mtp_destroy);
 *   - a 256-byte device status word of its own (see mtp_status_read).
 * mtp_context_bytes reports their size (about 6.3 GB for the full-shape
 * bf16 model).  Synchronises the device once (the repacking).  Returns
 * MTP_EUNSUPPORTED for shapes the kernels do not cover (hidden % 64,
 * head_dim not 64 or 128, n_routed > 64, ...), MTP_EHIP when an allocation
 * or copy fails (nothing is left allocated). */
mtp_status mtp_create(const mtp_config* cfg, const mtp_weights* w, mtp_ctx** out /* (host) */);
void mtp_destroy(mtp_ctx* ctx);

/* Device bytes the context holds (RoPE table, packed weights, status word);
 * 0 for a NULL context. */
size_t mtp_context_bytes(const mtp_ctx* ctx);

/* Workspace bytes for steps over `batch` sequences with up to `rows`
 * rows per sequence (a step needs rows = k+1; prefill uses chunks of at
 * most `rows` rows). */
size_t mtp_workspace_bytes(const mtp_ctx* ctx, int32_t batch, int32_t rows);

/* Blocking read of the sticky device status (after the caller has
 * synchronised the stream the step ran on): the workspace's word when it
 * is set, else the context's own word (set by kv_commit_rollback, which
 * takes no workspace).  ws may be NULL: the context's word only. */
mtp_status mtp_status_read(const mtp_ctx* ctx, const void* ws, int32_t* status /* (host) */);
/* Enqueues a reset of the context's status word and (ws not NULL) the
 * workspace's to MTP_OK. */
mtp_status mtp_status_clear(const mtp_ctx* ctx, void* ws, void* stream);

/* Prefill (the step before the hot path): runs the verifier over n_rows
 * rows per sequence at positions 0..n_rows-1 -- row i is the token
 * tok[b][i], or when tok[b][i] < 0 the vision row vision[b][i] -- writes
 * their K/V, takes the greedy token of the last row, and fills the draft
 * cache in base form for rows 0..n_rows-2 (state b_p, input row p+1).
 * Leaves the step state for the first step:
 *   kv_len = n_rows, draft_len = n_rows-1, n_rows_out = 1,
 *   row_pos = n_rows-1, hid[b][0] = b_{n_rows-1}, next_tok[b][0] = pending[b]
 *   = the greedy token, out_tok[b][0] = that token, n_out = 1.
 * k is the draft depth the following steps use: hid is [B][k+1][H] f32,
 * next_tok [B][k+1]; tok is [B][n_rows]; vision [B][n_rows][H] (storage
 * dtype) or NULL when every tok >= 0; out_tok [B][max_out].  route_idx,
 * when not NULL, receives the top-k experts of every row and layer,
 * [L][B][n_rows][top_k] (for checks). */
mtp_status mtp_prefill(mtp_ctx* ctx, int32_t batch, int32_t k, int32_t n_rows, const int32_t* tok,
                       const void* vision, void* kv_cache, void* draft_kv, int32_t* kv_len,
                       int32_t* draft_len, float* hid, int32_t* next_tok, int32_t* n_rows_out,
                       int32_t* row_pos, int32_t* pending, int32_t* out_tok, int32_t max_out,
                       int32_t* n_out, int32_t* route_idx, void* ws, size_t ws_bytes,
                       void* stream);

/* Draft (state-shift equation).  Depth 1 runs the catch-up rows
 * i = 0..n_rows[b]-1 at positions row_pos[b]+i, each with state
 * hid[b][i] and next input next_tok[b][i]; their draft K/V are written in
 * base form and the last row's LM-head argmax is draft_tok[b][0].  Depth
 * d = 2..k runs one row at position row_pos[b]+n_rows[b]-1+(d-1) with the
 * previous depth's output state and token.  Sets draft_len[b] =
 * row_pos[b]+n_rows[b].  Requires row_pos[b] <= draft_len[b] on entry
 * (device check).  draft_logits [B][k][V] f32 or NULL; draft_u [B][k][H]
 * f32 or NULL: the output state u of each depth (the state the next depth
 * starts from; for checks).  k = 0: no-op. */
mtp_status mtp_draft_k(mtp_ctx* ctx, int32_t batch, int32_t k, const float* hid,
                       const int32_t* next_tok, const int32_t* n_rows, const int32_t* row_pos,
                       void* draft_kv, int32_t* draft_len, int32_t* draft_tok,
                       float* draft_logits, float* draft_u, void* ws, size_t ws_bytes,
                       void* stream);

/* Verify: rows i = 0..k of sequence b hold pending[b] (i = 0) then
 * draft_tok[b][i-1], at positions kv_len[b]+i.  Writes their K/V in place,
 * runs the verifier, and returns verify_tok [B][k+1] (greedy token of each
 * row), hid [B][k+1][H] (final-norm state b of each row), and optionally
 * logits [B][k+1][V], margin [B][k+1] (top-1 minus top-2 logit),
 * route_idx [L][B*(k+1)][top_k], route_gap [L][B*(k+1)] (k-th minus
 * (k+1)-th router logit) and layer_h [L+1][B*(k+1)][H] f32 (the residual
 * stream entering layer l, and at l = L the last layer's output before the
 * final norm; for checks).  Row r of the routing and layer outputs is
 * sequence r / (k+1), row r % (k+1).  kv_len is not changed. */
mtp_status moe_verify_step(mtp_ctx* ctx, int32_t batch, int32_t k, const int32_t* pending,
                           const int32_t* draft_tok, const int32_t* kv_len, void* kv_cache,
                           int32_t* verify_tok, float* hid, float* logits, float* margin,
                           int32_t* route_idx, float* route_gap, float* layer_h, void* ws,
                           size_t ws_bytes, void* stream);

/* For callers that cannot allocate (code under HIP graph capture, serving
 * loops, harnesses that forbid hipMalloc): moe_verify_step with the same
 * arguments, outputs and kernels, but no workspace -- its scratch is a
 * static 16 MiB device array inside the library, one per device, looked up
 * and zero-filled by the first mtp_create on that device.  The call
 * allocates nothing.  Device conditions set the context's status word
 * (mtp_status_read with ws = NULL).  A batch whose scratch
 * (mtp_workspace_bytes(ctx, batch, k+1)) exceeds 16 MiB returns
 * MTP_EUNSUPPORTED and enqueues nothing (at the full shape: up to 16 rows,
 * batch x (k+1) <= 16, at any max_ctx).  Every call on a device shares that
 * device's scratch: calls that overlap in time on one device race and must
 * be ordered (one stream, or events); counters in it are left at zero by
 * each call and the array keeps the last call's contents. */
mtp_status moe_verify_step_static(mtp_ctx* ctx, int32_t batch, int32_t k,
                                  const int32_t* pending, const int32_t* draft_tok,
                                  const int32_t* kv_len, void* kv_cache, int32_t* verify_tok,
                                  float* hid, float* logits, float* margin, int32_t* route_idx,
                                  float* route_gap, float* layer_h, void* stream);

/* FastMTP draft-head objective, forward only (Section "Draft-head
 * objective", Eq. draft-loss and Eq. objective, over the training grid of
 * Section "Draft-head architecture").  One sequence of n_rows rows: row p
 * is the token tok[p], or when tok[p] < 0 the vision row vision[p]
 * ([n_rows][H] storage dtype; NULL when every tok >= 0); b_states
 * [n_rows][H] f32 are the verifier's post-norm states b_p (detached inputs,
 * e.g. from a verifier pass over the rows).  For each depth d = 1..k the
 * draft block runs over rows p = 0..n_rows-2 (next input row p+1,
 * position p, causal attention among the rows of that depth in its own
 * draft cache: draft_kv is [k][2][nh][max_ctx][dh], overwritten) with state
 * b_p at depth 1 and on prompt rows p < n_prompt, else u_{p-1}^(d-1).
 * Loss rows are p = n_prompt..n_rows-3 (response rows with a target
 * x_{p+2}; every target must be a token).  Outputs (device):
 *   loss [3k+1] f64: the means over the loss rows of CE_d, KL_d(Q||P),
 *     MSE_d for d = 1..k, then L = sum_d alpha_d (0.85 CE_d + 0.45 KL_d
 *     + 0.45 MSE_d), alpha_d = 0.6^(d-1) / sum_r 0.6^(r-1);
 *   row_terms [k][n_rows][3] f32 or NULL: each row's (CE, KL, MSE), zero
 *     outside the loss rows;
 *   u_out [k][n_rows][H] f32 or NULL: the draft outputs u_p^(d) (row
 *     n_rows-1 zero; for checks).
 * Requires 1 <= n_prompt <= n_rows - 3, n_rows <= max_ctx, 1 <= k <= 8 and
 * a workspace of mtp_objective_workspace_bytes(ctx, n_rows) bytes; device
 * conditions set the workspace's status word (MTP_ETOKEN for a target or
 * input outside the vocabulary). */
size_t mtp_objective_workspace_bytes(const mtp_ctx* ctx, int32_t n_rows);
mtp_status mtp_objective(mtp_ctx* ctx, int32_t n_rows, int32_t n_prompt, int32_t k,
                         const int32_t* tok, const void* vision, const float* b_states,
                         void* draft_kv, float* row_terms, float* u_out, double* loss, void* ws,
                         size_t ws_bytes, void* stream);

/* Acceptance equation: accept_len[b] = m, the longest r <= k with
 * draft_tok[b][s] == verify_tok[b][s] for all s < r; commit_tok[b] =
 * [draft_tok[b][0..m-1], verify_tok[b][m]] followed by -1 padding to k+1. */
mtp_status greedy_accept(int32_t batch, int32_t k, const int32_t* draft_tok,
                         const int32_t* verify_tok, int32_t* accept_len, int32_t* commit_tok,
                         void* stream);

/* Commit / rollback for each unfinished sequence (n_out[b] < limit, limit
 * = min(max_new[b], max_out), max_new NULL = max_out) whose accept_len[b]
 * lies in [0, k] (otherwise the context's status word is set to MTP_ERANGE
 * and the sequence is left unchanged):
 *   n_rows[b] = m+1, row_pos[b] = kv_len[b], kv_len[b] += m+1,
 *   pending[b] = commit_tok[b][m], next_tok[b][0..m] = commit_tok[b][0..m],
 *   out_tok[b][n_out..] += the committed tokens (truncated at the limit).
 * Finished sequences are left unchanged.  Rejected K/V rows need no
 * action: they lie at positions >= the new kv_len. */
mtp_status kv_commit_rollback(mtp_ctx* ctx, int32_t batch, int32_t k, const int32_t* accept_len,
                              const int32_t* commit_tok, int32_t* kv_len, int32_t* n_rows,
                              int32_t* row_pos, int32_t* pending, int32_t* next_tok,
                              const int32_t* max_new, int32_t* out_tok, int32_t max_out,
                              int32_t* n_out, void* stream);

/* Benchmark harness only (forced acceptance; not part of the method):
 * copies table[step][b][0..k-1] into draft_tok, step = *step_ctr, then
 * increments *step_ctr (wrapping at n_steps). */
mtp_status mtp_bench_override_drafts(int32_t batch, int32_t k, const int32_t* table,
                                     int32_t n_steps, int32_t* step_ctr, int32_t* draft_tok,
                                     void* stream);

/* Measurement only (not part of the method): per-launch timing of one
 * kernel class.  Between mtp_timing_start and mtp_timing_stop, every
 * launch of the class made by this context's calls is bracketed by a pair
 * of HIP events recorded on the call's stream (at most max_launches
 * launches; later ones are not timed).  Do not start timing while a stream
 * is being captured into a graph.  Timed launches are made with
 * hipExtLaunchKernelGGL, whose event pair the runtime stamps at the start
 * and the end of the dispatch itself.  mtp_timing_stop waits for the last
 * event and returns the summed launch durations (ms) and the number of
 * timed launches.  The context creates and destroys the events itself.
 * Errors: MTP_EINVAL (bad class, max_launches < 1, already started / not
 * started), MTP_EHIP. */
typedef enum {
  MTP_KC_ATTN = 1,       /* decode attention, split-K with fused merge */
  MTP_KC_MOE_GU = 2,     /* verifier MoE gate/up + SwiGLU (routed + shared) */
  MTP_KC_MOE_DOWN = 3,   /* verifier MoE down projection */
  MTP_KC_LM_HEAD = 4,    /* LM head partial argmax (verifier and draft) */
  MTP_KC_QKV = 5,        /* fused RMSNorm + QKV + RoPE + K/V append */
  MTP_KC_ROUTER = 6,     /* fused RMSNorm + router + top-k */
  MTP_KC_DRAFT_FFN = 7,  /* draft block FFN gate/up + SwiGLU */
  MTP_KC_MOE = 8         /* verifier MoE sub-layer of up to 16 rows in one launch
                            (RMSNorm + router + top-k, gate/up + SwiGLU, down) */
} mtp_kernel_class;
mtp_status mtp_timing_start(mtp_ctx* ctx, int32_t kernel_class, int32_t max_launches);
mtp_status mtp_timing_stop(mtp_ctx* ctx, float* total_ms /* (host) */,
                           int32_t* n_launches /* (host) */);

#ifdef __cplusplus
}
#endif
#endif /* MTP_H */
