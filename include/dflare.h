/*
 * dflare.h -- C ABI of the DFlare draft step on AMD Instinct MI355X (gfx950).
 *
 * The library computes the per-iteration draft step of DFlare (arXiv 2606.02091):
 *   - layer fusion: each draft layer i fuses the hidden rows of S target layers
 *     with its own softmax weights, alpha^(i) = softmax(W^fuse_{i,:}), then RMSNorm
 *     (Sec. 4.1, Eq. 3; alpha is computed once at init, as Sec. 4.1 allows);
 *   - heterogeneous context K/V: the fused rows of layer i go through that layer's
 *     own W_K^t, W_V^t into its KV cache (Sec. 4.2, Eq. 4, first block);
 *   - the drafting forward pass: the B block rows [x_t; mask x (B-1)] run through
 *     D draft layers with block K/V from W_K^d, W_V^d (Eq. 4, other blocks),
 *     attention that is bidirectional inside the block and sees the whole context,
 *     an MLP sub-layer, then the shared LM head and one token per position
 *     (Sec. 3.2, drafting phase).
 *
 * Readings where the paper is silent: pre-norm layers with residuals around
 * attention and MLP, SwiGLU MLP, no biases, final RMSNorm before the LM head,
 * RMSNorm(x; g) = x / sqrt(mean(x^2) + eps) * g, rotary embedding in the
 * rotate-half convention (context keys rotated at their own positions when
 * appended), context row r at position r and block row b at position L + b,
 * scale 1/sqrt(head_dim), query head h uses KV head h / (n_q / n_kv), greedy
 * argmax with ties to the lowest id unless dflare_set_sampling sets a temperature.
 *
 * Conventions for every entry point:
 *   - Return value: DFLARE_OK (0) or a negative dflare_status.  Nothing throws.
 *   - Arguments are validated before any work is enqueued; a call that fails
 *     validation changes no state (context length, cache, handle).
 *   - Device pointers are borrowed: the caller keeps ownership and must keep them
 *     valid until the work enqueued on the handle's stream has completed.
 *   - Work is enqueued on the handle's stream and the call returns without
 *     waiting (except where stated).  Results are valid once that stream is
 *     synchronised.
 *   - A handle is not thread-safe: calls on one handle must not overlap.
 *   - bf16 means IEEE-754 binary32 truncated to its upper 16 bits (bfloat16),
 *     passed as raw 16-bit patterns.
 */
#ifndef DFLARE_H
#define DFLARE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DFLARE_OK = 0,
  DFLARE_ERR_INVALID_ARG = -1,   /* bad pointer, size, shape or value            */
  DFLARE_ERR_OUT_OF_MEMORY = -2, /* device allocation failed                      */
  DFLARE_ERR_CONTEXT_FULL = -3,  /* append would exceed max_context               */
  DFLARE_ERR_HIP = -4,           /* a HIP runtime call failed                     */
  DFLARE_ERR_UNSUPPORTED = -5    /* shape the kernels do not support (see init)   */
} dflare_status;

/* Model and capacity.  All sizes are element counts. */
typedef struct {
  int32_t hidden;          /* H (the paper's d)                                  */
  int32_t n_q_heads;       /* query heads                                        */
  int32_t n_kv_heads;      /* key/value heads (n_q_heads % n_kv_heads == 0)      */
  int32_t head_dim;        /* per-head width                                     */
  int32_t ffn;             /* SwiGLU inner width                                 */
  int32_t vocab;           /* V                                                  */
  int32_t n_draft_layers;  /* D                                                  */
  int32_t n_target_layers; /* S (the paper's T), fused target layers             */
  int32_t block_size;      /* B, 1..16                                           */
  int32_t max_context;     /* L_max: capacity of the per-layer context cache     */
  int32_t max_new;         /* largest n_new accepted by dflare_fuse_append       */
  float rope_base;         /* rotary base, e.g. 1e6                              */
  float rms_eps;           /* RMSNorm epsilon, e.g. 1e-6                         */
  int32_t max_batch;       /* sequence slots for the batched calls, 1..64
                              (0 means 1); slot 0 is the batch-1 context         */
  int32_t variant;         /* 0, or DFLARE_VARIANT_* flags (below)               */
} dflare_config;

/*
 * Model variants (dflare_config.variant; 0 is the method as described).  They change
 * only how appended target rows become context K/V (dflare_fuse_append and its
 * batched form); the draft block is the same for all of them.
 *   NO_SOFTMAX  the -Softmax ablation (Sec. 6.3, Table 2): alpha = W^fuse as given,
 *               every entry finite.
 *   SHARED_KV   the -KVProj ablation (Sec. 6.3): the fused context goes through each
 *               layer's own W_K^d, W_V^d; wk_t and wv_t are not read (may be NULL).
 *   POST_FC     the +FC ablation (Sec. 6.3): f' = f W_pfc^T + b_pfc on each layer's
 *               fused rows before its context projection (weights post_fc,
 *               post_fc_bias).  The library folds the layer into the projection at
 *               init: W' = W_K W_pfc and b' = W_K b_pfc (likewise for V) in double
 *               precision, W' rounded to bf16, b' kept in fp32.
 *   DFLASH      the DFlash baseline (Sec. 3.1-3.2, Eq. 1-2): one context row
 *               c_t = W_fc [h_t^(1); ...; h_t^(S)] + b_fc (weights fc, fc_bias) for
 *               every draft layer, projected by the layer's W_K^d, W_V^d; no fusion
 *               weights (fusion_logits may be NULL) and no fusion norm.  The append
 *               runs on fp16 matrix-core operands (target rows saturated to +-65504).
 *               Not combinable with the other flags.
 */
#define DFLARE_VARIANT_NO_SOFTMAX 1
#define DFLARE_VARIANT_SHARED_KV 2
#define DFLARE_VARIANT_POST_FC 4
#define DFLARE_VARIANT_DFLASH 8

/*
 * Draft weights: device pointers to bf16 tensors, row-major, linear weights in the
 * [out, in] convention (y = x W^T), stacked over the D draft layers.
 * q = n_q_heads * head_dim, kv = n_kv_heads * head_dim.
 * A NULL norm gain means all ones.  Init copies and re-packs everything, so the
 * caller may free these buffers once dflare_init has returned.
 */
typedef struct {
  const void* embed;      /* [V, H]     shared token embedding (Sec. 3.3)       */
  const void* lm_head;    /* [V, H]     shared LM head (Sec. 3.3)               */
  const void* final_norm; /* [H]        gain of the final RMSNorm, or NULL      */
  const void* fuse_norm;  /* [D, H]     gain of the RMSNorm in Eq. 3, or NULL   */
  const void* attn_norm;  /* [D, H]     pre-attention RMSNorm gain, or NULL     */
  const void* mlp_norm;   /* [D, H]     pre-MLP RMSNorm gain, or NULL           */
  const void* wq;         /* [D, q, H]  W_Q                                     */
  const void* wk_d;       /* [D, kv, H] W_K^d (block rows, Eq. 4)               */
  const void* wv_d;       /* [D, kv, H] W_V^d                                   */
  const void* wk_t;       /* [D, kv, H] W_K^t (fused target context, Eq. 4)     */
  const void* wv_t;       /* [D, kv, H] W_V^t                                   */
  const void* wo;         /* [D, H, q]  attention output projection             */
  const void* w_gate;     /* [D, F, H]  SwiGLU gate                             */
  const void* w_up;       /* [D, F, H]  SwiGLU up                               */
  const void* w_down;     /* [D, H, F]  SwiGLU down                             */
  /* variant weights, read only by the variants that use them (NULL otherwise)    */
  const void* post_fc;      /* [D, H, H]   POST_FC: W_pfc per draft layer        */
  const void* post_fc_bias; /* [D, H]      POST_FC: b_pfc, or NULL for zeros      */
  const void* fc;           /* [H, S*H]    DFLASH: W_fc (Eq. 1), input = the S
                                           rows of a position in layer order      */
  const void* fc_bias;      /* [H]         DFLASH: b_fc, or NULL for zeros        */
} dflare_weights;

typedef struct dflare_handle dflare_handle;

/*
 * dflare_init -- build a draft model (Sec. 4.1 Eq. 3, Sec. 4.2 Eq. 4, Sec. 3.2).
 *   cfg            model shape and capacity.  Supported: hidden, q and ffn
 *                  multiples of 32, hidden <= 8192; head_dim 64 or 128;
 *                  1 <= block_size <= 16; (n_q_heads / n_kv_heads) * block_size
 *                  <= 128; n_target_layers <= 64; otherwise DFLARE_ERR_UNSUPPORTED.
 *   weights        device bf16 tensors as described above (copied and packed).
 *   fusion_logits  HOST float [D, S] = W^fuse.  alpha = softmax of each row is
 *                  computed here in double precision and cached as float.  A row
 *                  with NaN or +inf, or with no finite entry, is INVALID_ARG.
 *                  Unused (may be NULL) with DFLARE_VARIANT_DFLASH; taken as alpha
 *                  itself with DFLARE_VARIANT_NO_SOFTMAX.
 *   A variant value with unknown bits, DFLASH combined with another flag, or a
 *   missing weight that the variant reads is INVALID_ARG.
 *   stream         hipStream_t for all work of this handle (NULL = default stream).
 *   out            receives the handle.  Every context starts empty (L = 0).
 * Each of the max_batch sequence slots owns a context cache of max_context rows
 * per draft layer.
 * Synchronises the stream before returning.
 */
int dflare_init(const dflare_config* cfg, const dflare_weights* weights,
                const float* fusion_logits, void* stream, dflare_handle** out);

/*
 * dflare_fuse_append -- fuse n_new accepted target rows and append their K/V
 * to every draft layer's cache (Sec. 4.1 Eq. 3, Sec. 4.2 Eq. 4 first block).
 *   target_hidden  DEVICE bf16 [S, n_new, H] (target layer major).  Row r of the
 *                  call becomes context position L + r.
 *   n_new          1 <= n_new <= max_new, else INVALID_ARG;
 *                  L + n_new > max_context gives CONTEXT_FULL and changes nothing.
 * On success L grows by n_new.
 */
int dflare_fuse_append(dflare_handle* h, const void* target_hidden, int32_t n_new);

/*
 * dflare_accept -- the verification step of the draft-then-verify loop (Sec. 3.2,
 * verification phase) on slot 0, with the target's outputs computed by the caller.
 *   block_ids      DEVICE int32 [B]: the drafted block (x_t at 0, mask ids at 1..B-1).
 *   draft_tokens   DEVICE int32 [B]: dflare_draft_block's output for it (candidates
 *                  at 1..B-1).
 *   target_tokens  DEVICE int32 [B]: the target's own next token after each block
 *                  position b (given x_t and candidates 1..b).
 *   target_hidden  DEVICE bf16 [S, B, H]: the target's hidden rows at the B positions.
 *   next_ids       DEVICE int32 [B], out: the next block -- the bonus token, then
 *                  block_ids[1..B-1].  May be block_ids itself (updated in place).
 *   emitted        DEVICE int32 [B], out: the k accepted candidates, the bonus token,
 *                  then -1 (k + 1 tokens: what the target alone would emit greedily).
 *   accepted       HOST int32 out, or NULL: k.
 * k is the number of leading candidates j = 1.. equal to the target's token after
 * position j - 1 (0 <= k <= B-1); the bonus token is the target's token after
 * position k.  The target rows of positions 0..k (x_t and the accepted candidates) are
 * appended to the context as dflare_fuse_append would (L grows by k + 1), selected and
 * fused on the device.  The call waits for the stream once, after the selection, so
 * that the host knows k and the new L.  max_new < B: INVALID_ARG; L + B > max_context:
 * CONTEXT_FULL, and nothing changes.
 */
int dflare_accept(dflare_handle* h, const int32_t* block_ids, const int32_t* draft_tokens,
                  const int32_t* target_tokens, const void* target_hidden, int32_t* next_ids,
                  int32_t* emitted, int32_t* accepted);

/*
 * dflare_accept_async -- dflare_accept without the wait (Sec. 3.2, verification phase):
 * the whole draft-then-verify loop stays on the stream, the host never learns k.
 *   block_ids .. emitted   as for dflare_accept.
 *   accepted_dev   DEVICE int32 out, or NULL: k.
 * The new context length L + k + 1 is kept on the device, and the next dflare_draft_block
 * and dflare_accept_async read it there.  All B target rows are fused and their K/V written
 * to slots L .. L + B - 1; the k + 1 verified ones become the context, the others lie past
 * it and are overwritten by the next draft block's own keys before anything reads them.
 * Every other call that needs L (dflare_context_len, dflare_truncate, dflare_fuse_append,
 * dflare_accept, dflare_draft_block_pos, the batched and debug calls) first waits for the
 * stream and takes the length back to the host.  The host keeps an upper bound (L + B per
 * call); when the bound leaves no room for B more rows it reads the length first, and
 * L + B > max_context then gives CONTEXT_FULL with nothing changed.  max_new < B:
 * INVALID_ARG.  For the DFlash variant (whose fusion takes host lengths) the call waits as
 * dflare_accept does.
 */
int dflare_accept_async(dflare_handle* h, const int32_t* block_ids, const int32_t* draft_tokens,
                        const int32_t* target_tokens, const void* target_hidden, int32_t* next_ids,
                        int32_t* emitted, int32_t* accepted_dev);

/*
 * dflare_draft_block -- one drafting forward pass (Sec. 3.2, drafting phase).
 *   block_ids      DEVICE int32 [B]: x_t at index 0, the mask id at 1..B-1 (the
 *                  library treats all ids alike; ids outside [0, V) are clamped).
 *   draft_tokens   DEVICE int32 [B]: token at every block position (greedy, or sampled
 *                  as dflare_set_sampling sets, in sequence slot 0); index 0 is not a
 *                  candidate (the B-1 candidates are 1..B-1).
 * Block row b sits at position L + b.  The context cache is not modified, so the
 * call can be repeated.  An empty context (L = 0) is allowed.
 * By default the whole pass is one launch of one work-group per CU whose phases
 * are separated by grid barriers or per-KV-head counters (see
 * DFLARE_OPT_PERSISTENT); these waits need every work-group resident at once
 * (DFLARE_OPT_COOPERATIVE).  If a grid barrier
 * of an earlier call timed out (the work-groups were not all resident within
 * 0.25 s), this call returns DFLARE_ERR_HIP without enqueuing work and the handle
 * switches to one launch per phase.
 */
int dflare_draft_block(dflare_handle* h, const int32_t* block_ids, int32_t* draft_tokens);

/*
 * dflare_draft_block_pos -- as dflare_draft_block, with explicit block positions
 * (a test entry for position-dependent invariants).
 *   positions      HOST int32 [B], each in [0, max_context + block_size).
 */
int dflare_draft_block_pos(dflare_handle* h, const int32_t* block_ids, const int32_t* positions,
                           int32_t* draft_tokens);

/* dflare_truncate -- roll the context back to new_len (0 <= new_len <= L). */
int dflare_truncate(dflare_handle* h, int32_t new_len);

/* dflare_context_len -- current context length L into *out (waits for the stream when the
 * length is on the device, after dflare_accept_async). */
int dflare_context_len(const dflare_handle* h, int32_t* out);

/*
 * Batched calls: the draft step of several independent sequences at once (Sec. 3.2
 * drafting phase and Sec. 4.1-4.2 context update, applied per sequence; the
 * sequences share the draft weights and nothing else).  Sequence slots are
 * 0 .. max_batch-1, each with its own context length and cache; the batch-1 calls
 * above work on slot 0.  In every batched call:
 *   n_seq          1 <= n_seq <= max_batch
 *   seq            HOST int32 [n_seq]: distinct slots in [0, max_batch)
 * Results are those of the batch-1 calls on each slot in turn, up to rounding
 * order: the batched kernels sum in a different order (same precision).
 */

/*
 * dflare_fuse_append_batched -- dflare_fuse_append for sequence seq[i] with
 * n_new[i] rows, for every i.
 *   n_new          HOST int32 [n_seq], each >= 1, sum <= max_new, else INVALID_ARG;
 *                  L_seq[i] + n_new[i] > max_context for any i gives CONTEXT_FULL
 *                  and changes nothing.
 *   target_hidden  DEVICE bf16 [S, sum(n_new), H]: for each target layer, the rows
 *                  of seq[0], then those of seq[1], ...
 */
int dflare_fuse_append_batched(dflare_handle* h, int32_t n_seq, const int32_t* seq, const int32_t* n_new,
                               const void* target_hidden);

/*
 * dflare_draft_block_batched -- dflare_draft_block for every listed sequence.
 *   block_ids      DEVICE int32 [n_seq, B]: row i is the block of seq[i].
 *   draft_tokens   DEVICE int32 [n_seq, B]: tokens (greedy, or sampled as dflare_set_sampling
 *                  sets), row i for seq[i].
 * Block row b of seq[i] sits at position L_seq[i] + b.  No cache is modified.
 */
int dflare_draft_block_batched(dflare_handle* h, int32_t n_seq, const int32_t* seq, const int32_t* block_ids,
                               int32_t* draft_tokens);

/*
 * dflare_set_sampling -- how draft tokens are chosen from the logits z (Sec. 3.2 samples the
 * candidates; the paper reports greedy and temperature-1 decoding, Sec. 5, Table 1).
 *   temperature    0 (the default): greedy argmax, ties to the lowest id.  > 0: each position's
 *                  token is argmax_v (z_v / temperature + G_v) with Gumbel noise
 *                  G_v = -log(-log(U_v)), a draw from softmax(z / temperature).  Negative,
 *                  NaN, infinite, or so small that 1 / temperature overflows fp32: INVALID_ARG.
 *   seed           key of the noise.  U_v at block position b = (top 23 bits of word b mod 4 of
 *                  Philox4x64-10 (Salmon et al., SC 2011) at counter (v, b div 4, draw, sequence
 *                  slot) under key (seed, 0) + 1/2) / 2^23, exact in fp32; draw counts the draft
 *                  calls (batch-1 or batched) made since this call, from 0.  The batch-1 calls use
 *                  slot 0.
 * Debug logits stay the unperturbed z.  Takes effect for later draft calls.
 */
int dflare_set_sampling(dflare_handle* h, float temperature, uint64_t seed);

/* dflare_truncate_seq / dflare_context_len_seq -- as above, for one slot. */
int dflare_truncate_seq(dflare_handle* h, int32_t seq, int32_t new_len);
int dflare_context_len_seq(const dflare_handle* h, int32_t seq, int32_t* out);

/* dflare_set_stream -- make later work of the handle go to `stream`. */
int dflare_set_stream(dflare_handle* h, void* stream);

/* dflare_destroy -- free the handle and everything it owns (synchronises). */
int dflare_destroy(dflare_handle* h);

/* Status code -> static string. */
const char* dflare_status_str(int status);

/* Last error message of the handle (static empty string when none or h is NULL). */
const char* dflare_last_error(const dflare_handle* h);

/*
 * Debug capture (tests).  While on, draft_block keeps the block rows after each
 * layer and the full logits, and fuse_append keeps the fused rows f^(i).
 * dflare_debug_read synchronises the stream and copies one tensor to HOST float:
 *   what = DFLARE_DBG_FUSED   layer i: [n_last, H]   fused rows f^(i) of the last append
 *   what = DFLARE_DBG_KCACHE  layer i: [L, n_kv, hd] context keys (after RoPE)
 *   what = DFLARE_DBG_VCACHE  layer i: [L, n_kv, hd] context values
 *   what = DFLARE_DBG_HIDDEN  layer i: [B, H]        block rows after layer i
 *   what = DFLARE_DBG_LOGITS  (layer ignored) [B, V] logits of the last draft_block
 *   what = DFLARE_DBG_ALPHA   (layer ignored) [D, S] cached fusion weights
 *   what = DFLARE_DBG_BLOGITS (layer ignored) [n_seq, B, V] logits of the last
 *                             dflare_draft_block_batched (n_seq of that call)
 *   what = DFLARE_DBG_TRACE   (layer ignored) [blocks, phases, 4] microseconds, relative to
 *                             the earliest mark, at which each work-group of the last
 *                             draft_block reached four marks of each phase: body start
 *                             (after its grid barrier), two inner marks (GEMM phases: main
 *                             loop done, chunk epilogues done; attention: keys staged in LDS,
 *                             scores and values done), stores complete; -1 where a phase sets
 *                             no such mark.  Needs DFLARE_OPT_TRACE (sizes from
 *                             dflare_kernel_stats)
 * `count` is the number of floats host_out can hold; too small is INVALID_ARG.
 * Debug capture makes draft_block run one launch per phase, unless
 * DFLARE_OPT_CAPTURE_PERSISTENT is set.  FUSED after a
 * batched append holds all sum(n_new) rows of that call.
 * dflare_debug_read_seq reads DFLARE_DBG_KCACHE / DFLARE_DBG_VCACHE of slot `seq`
 * ([L_seq, n_kv, hd]); dflare_debug_read reads those of slot 0.
 */
enum { DFLARE_DBG_FUSED = 0, DFLARE_DBG_KCACHE = 1, DFLARE_DBG_VCACHE = 2,
       DFLARE_DBG_HIDDEN = 3, DFLARE_DBG_LOGITS = 4, DFLARE_DBG_ALPHA = 5,
       DFLARE_DBG_TRACE = 6, DFLARE_DBG_BLOGITS = 7 };
int dflare_debug_capture(dflare_handle* h, int on);
int dflare_debug_read(dflare_handle* h, int what, int layer, float* host_out, int64_t count);
int dflare_debug_read_seq(dflare_handle* h, int what, int seq, int layer, float* host_out, int64_t count);

/*
 * dflare_kernel_stats -- launch shape, for measurement: writes up to `count`
 * int32 values
 *   [0] number of kernels one draft_block enqueues
 *   [1] number of kernels one fuse_append enqueues
 *   [2] work-groups of the draft-block kernel
 *   [3] phases of a draft block (embedding; per layer QKV, attention, combine,
 *       output projection, gate/up, down; LM head)
 *   [4] grid barriers one draft_block waits at (0 with one launch per phase; the
 *       attention and combine phases wait for their KV head's Q/K/V tiles and
 *       attention items instead)
 *   [5] plan signature of the draft-block kernel that runs: the chunk widths of
 *       the Q/K/V, output, gate/up and down GEMMs in 4 bits each (Q/K/V lowest) for
 *       a kernel built for the handle's plans, 0 for the generic kernel
 */
int dflare_kernel_stats(const dflare_handle* h, int32_t* out, int32_t count);

/*
 * Kernel timing (measurement).  dflare_profile_begin(h, kind) brackets every later
 * launch of one kernel kind with a pair of hipEvents on the handle's stream, up to
 * 8192 launches; kind = 0 stops.  dflare_profile_end synchronises the stream and
 * returns the summed event-measured duration (ms) and the number of launches
 * timed since the last begin, then stops.  Kinds 1-6 are phases of the draft
 * block: while one of them is profiled, draft_block runs one launch per phase.
 * Kinds:
 */
enum { DFLARE_K_QKV = 1,       /* RMSNorm + Q/K^d/V^d projection + RoPE           */
       DFLARE_K_ATTN = 2,      /* block attention (split over keys) + combine      */
       DFLARE_K_O = 3,         /* output projection + residual                     */
       DFLARE_K_GATE_UP = 4,   /* RMSNorm + gate/up projection + SwiGLU            */
       DFLARE_K_DOWN = 5,      /* down projection + residual                       */
       DFLARE_K_LM_HEAD = 6,   /* final RMSNorm + LM head + argmax                 */
       DFLARE_K_FUSE = 7,      /* layer fusion (Eq. 3)                             */
       DFLARE_K_KV_T = 8,      /* context K/V projection + RoPE + append (Eq. 4)   */
       DFLARE_K_DRAFT = 9,     /* a whole draft_block, as configured               */
       /* batched calls */
       DFLARE_K_B_QKV = 10,    /* Q/K^d/V^d projection GEMM                        */
       DFLARE_K_B_ATTN = 11,   /* attention over every sequence + combine          */
       DFLARE_K_B_O = 12,      /* output projection GEMM                           */
       DFLARE_K_B_GATE_UP = 13,/* gate/up projection GEMM                          */
       DFLARE_K_B_DOWN = 14,   /* down projection GEMM                             */
       DFLARE_K_B_LM_HEAD = 15,/* LM-head GEMM with partial argmax + final argmax  */
       DFLARE_K_B_KV_T = 16,   /* context K/V projection GEMM of an append         */
       DFLARE_K_B_EPI = 17,    /* embedding, row norms and GEMM epilogues          */
       DFLARE_K_B_FUSE = 18,   /* layer fusion of an append                        */
       DFLARE_K_B_DRAFT = 19,  /* a whole dflare_draft_block_batched               */
       DFLARE_K_B_APPEND = 20 };/* a whole dflare_fuse_append_batched              */
int dflare_profile_begin(dflare_handle* h, int kind);
int dflare_profile_end(dflare_handle* h, double* total_ms, int32_t* launches);

/*
 * dflare_set_option -- execution options of a handle (they do not change results):
 *   DFLARE_OPT_PERSISTENT  1 (default): a draft_block is one launch whose phases wait
 *                          at grid barriers; 0: one launch per phase.  1 is refused
 *                          (UNSUPPORTED) when the device cannot keep one work-group per
 *                          CU resident.
 *   DFLARE_OPT_COOPERATIVE 0 (default): the persistent launch is a plain launch of one
 *                          work-group per CU (each takes a whole CU's LDS).  The stream's
 *                          earlier work has ended when it starts, so all work-groups are
 *                          placed at once unless kernels of other streams or processes
 *                          hold CUs; those delay the late work-groups until they end, and
 *                          past 0.25 s at a barrier the call fails as described under
 *                          dflare_draft_block.  1: a cooperative launch, for which the
 *                          runtime guarantees co-residency, at about 13 us more per call
 *                          (it is ordered against the device's other queues).
 *   DFLARE_OPT_TRACE       1: record per-work-group phase start times (DFLARE_DBG_TRACE).
 *   DFLARE_OPT_CAPTURE_PERSISTENT
 *                          1: debug capture keeps the persistent launch: the draft-block
 *                          kernel itself writes the logits and the block rows after each
 *                          layer (DFLARE_DBG_LOGITS, DFLARE_DBG_HIDDEN) in the launch
 *                          configuration that is timed; 0 (default): debug capture runs
 *                          one launch per phase.
 *   DFLARE_OPT_GENERIC_KERNEL
 *                          0 (default): where the library holds a draft-block kernel built
 *                          for the handle's GEMM plans (the plans chosen for the Qwen3-8B,
 *                          Qwen3-4B and GPT-OSS-20B shapes on 256 CUs), that kernel runs;
 *                          1: the generic kernel, which reads the plans at run time.  Both
 *                          compute the same results bit for bit.
 */
enum {
  DFLARE_OPT_PERSISTENT = 1,
  DFLARE_OPT_TRACE = 2,
  DFLARE_OPT_CAPTURE_PERSISTENT = 3,
  DFLARE_OPT_COOPERATIVE = 4,
  DFLARE_OPT_GENERIC_KERNEL = 5
};
int dflare_set_option(dflare_handle* h, int option, int value);

/*
 * dflare_read_probe -- measurement helper, no handle: one plain streaming read of `bytes`
 * (a positive multiple of 16) of DEVICE memory at `buf` with 16-byte nontemporal loads,
 * eight per thread in flight, on eight 256-thread work-groups per CU; `sink` is one DEVICE
 * uint32 that the kernel writes only in a case that practically never occurs.  The rate it
 * reaches is the HBM read ceiling the draft kernels are quoted against next to the 8 TB/s
 * specification.  Asynchronous on `stream` (NULL = default); INVALID_ARG on a bad argument.
 */
int dflare_read_probe(const void* buf, int64_t bytes, uint32_t* sink, void* stream);

/*
 * ---- Training-side kernels (no handle) ----
 * Anchor attention of one draft layer (Sec. 3.3): the n_blocks sampled blocks of one
 * training sequence are processed together; the rows of block i, anchored at sequence
 * position anchors[i] (0 <= anchors[i] <= T), attend to the target context features of the
 * positions before the anchor (context keys 0 .. anchors[i]-1) and bidirectionally to the B
 * positions of their own block; never to another block.  Scale 1/sqrt(hd); query head h
 * reads KV head h / (n_q / n_kv).  Rotary embedding, if any, is already applied.
 *   q              DEVICE bf16 [n_blocks*B, n_q, hd]   (row i*B + b: block i, position b)
 *   k_ctx, v_ctx   DEVICE bf16 [T, n_kv, hd]           (may be NULL when T = 0)
 *   k_blk, v_blk   DEVICE bf16 [n_blocks*B, n_kv, hd]
 *   anchors        DEVICE int32 [n_blocks]
 *   out            DEVICE fp32 [n_blocks*B, n_q, hd];  lse  DEVICE fp32 [n_blocks*B, n_q]
 *                  (natural log-sum-exp of each row's scaled scores, for the backward pass)
 *   workspace      DEVICE scratch of at least dflare_anchor_attention_workspace(...) bytes
 *                  (transposed copies and partial sums; contents need not be kept)
 * Supported: 1 <= B <= 16, hd 64 or 128, (n_q / n_kv) * B <= 128; else UNSUPPORTED.  The
 * products run on bf16 matrix cores (probabilities and gradients rounded to bf16 as operands,
 * fp32 accumulation).  Asynchronous on `stream` (hipStream_t, NULL = default).  Gradients are
 * deterministic: context-key gradients are summed over chunks of 64 blocks in a fixed order.
 */
size_t dflare_anchor_attention_workspace(int32_t n_blocks, int32_t B, int32_t T, int32_t n_q, int32_t n_kv,
                                         int32_t hd);
int dflare_anchor_attention_fwd(const void* q, const void* k_ctx, const void* v_ctx, const void* k_blk,
                                const void* v_blk, const int32_t* anchors, int32_t n_blocks, int32_t B, int32_t T,
                                int32_t n_q, int32_t n_kv, int32_t hd, float* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream);
/*
 * Backward of the above for the output gradient dout (DEVICE fp32 [n_blocks*B, n_q, hd]),
 * given the forward's out and lse: dq [n_blocks*B, n_q, hd], dk_ctx / dv_ctx [T, n_kv, hd],
 * dk_blk / dv_blk [n_blocks*B, n_kv, hd], all DEVICE fp32, overwritten.
 */
int dflare_anchor_attention_bwd(const void* q, const void* k_ctx, const void* v_ctx, const void* k_blk,
                                const void* v_blk, const int32_t* anchors, int32_t n_blocks, int32_t B, int32_t T,
                                int32_t n_q, int32_t n_kv, int32_t hd, const float* out, const float* lse,
                                const float* dout, float* dq, float* dk_ctx, float* dv_ctx, float* dk_blk,
                                float* dv_blk, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Progressive position-weighted cross-entropy (Sec. 4.3, Eq. 5) over rows = n_blocks * B
 * block positions: row r is position b = r % B of its block; the anchor position (b = 0)
 * and rows with label < 0 (or >= V) carry no loss; position b >= 1 has weight
 * w = exp(-(b - 1) / gamma), gamma = gamma(s) of the schedule (the caller's).  The loss is
 * sum w CE / sum w.
 *   logits   DEVICE fp32 [rows, V];  labels  DEVICE int32 [rows]
 *   loss     DEVICE fp32 [1] out;  row_ce  DEVICE fp32 [rows] out (CE per row, 0 where no loss)
 *   dlogits  DEVICE fp32 [rows, V] out: d loss / d logits
 *   workspace DEVICE scratch of at least dflare_weighted_ce_workspace(rows) bytes
 * rows not a multiple of B, gamma <= 0 or not finite: INVALID_ARG.  Deterministic.
 */
size_t dflare_weighted_ce_workspace(int32_t rows);
int dflare_weighted_ce(const float* logits, const int32_t* labels, int32_t rows, int32_t V, int32_t B, float gamma,
                       float* loss, float* row_ce, float* dlogits, void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * dflare_weighted_ce_noalloc -- the weighted CE above for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and kernels as dflare_weighted_ce, without the
 * workspace: the row weights and 1 / sum w live in a fixed device array of the library
 * (DFLARE_WEIGHTED_CE_NOALLOC_MAX_ROWS + 64 floats, 256 KiB + 256 B; each GPU the library
 * runs on holds its own copy until the process ends).  Calls no hipMalloc, hipFree or other
 * allocating routine.  rows > DFLARE_WEIGHTED_CE_NOALLOC_MAX_ROWS: INVALID_ARG; a non-NULL
 * `stream` must belong to the current device (else INVALID_ARG).  The array is shared by
 * every call on a GPU and keeps the last call's contents (each call writes every value it
 * reads before reading it): calls that overlap in time on one GPU (different streams, or
 * different host threads) race and give undefined results; calls ordered on one stream do
 * not.
 */
#define DFLARE_WEIGHTED_CE_NOALLOC_MAX_ROWS 65536
int dflare_weighted_ce_noalloc(const float* logits, const int32_t* labels, int32_t rows, int32_t V, int32_t B,
                               float gamma, float* loss, float* row_ce, float* dlogits, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DFLARE_H */
