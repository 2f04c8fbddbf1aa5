/*
 * dllm.h -- C ABI of the CAI-dLLM denoising-step library for MI355X (gfx950).
 *
 * One denoising step of a masked diffusion language model (Section 4.1 and
 * Algorithm 1 of the CAI-dLLM paper): a bidirectional transformer forward over
 * prompt + generated positions, a vocabulary-wide confidence / argmax
 * reduction at the current block's positions (Box 1), and the confidence-aware
 * commit rule (Boxes 2-7) that updates the decoding state in place.
 *
 * Conventions (every entry point):
 *  - Pointers documented "device" are HIP device memory owned by the caller;
 *    the library never frees them and keeps none after the call returns,
 *    except those a model handle borrows for its lifetime: the weights, the
 *    model buffer of dllm_model_create and the buffer of
 *    dllm_model_pack_weights.
 *  - The library allocates no device memory.  Every buffer is the caller's,
 *    sized by a query: the model buffer (dllm_model_buffer_size), the packed
 *    weights (dllm_model_packed_size), the workspace (dllm_workspace_size) and
 *    the key/value cache (dllm_kv_cache_size), each 256-byte aligned.  The
 *    only other resources are host objects of a model handle (one coherent
 *    pinned host word the commit kernel publishes each step's done flag to,
 *    timing events).
 *  - `stream` is a hipStream_t passed as void*; NULL is the null stream.  All
 *    device work is enqueued on it in order; entry points return once the work
 *    is enqueued unless stated otherwise.
 *  - Every function returns a dllm_status.  On failure nothing is enqueued
 *    (argument errors) or the HIP error is reported (DLLM_EHIP); the message of
 *    the last failure on the calling thread is returned by dllm_last_error().
 *  - Integer sizes are int32; B = batch, P = prompt length, G = generated
 *    length, L = P + G, bl = block length.
 *  - Not thread-safe per model handle: calls that share a model or a workspace
 *    must be ordered by the caller.
 */
#ifndef DLLM_H
#define DLLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dllm_status {
  DLLM_OK = 0,
  DLLM_EINVAL = -1,       /* invalid argument value (NaN threshold, null pointer, ...) */
  DLLM_ESHAPE = -2,       /* inconsistent sizes */
  DLLM_EHIP = -3,         /* a HIP runtime call failed */
  DLLM_ENOMEM = -4,       /* workspace too small */
  DLLM_EUNSUPPORTED = -5  /* valid but not implemented for this shape / dtype */
} dllm_status;

/* Storage type of weights and matrix-product operands. */
enum { DLLM_F32 = 0, DLLM_BF16 = 1 };

/*
 * Model shape.  The paper names its models (LLaDA-8B, Dream-7B; Section 5) but
 * prints no architecture: this is the pre-norm layer those models share
 * (RMSNorm, rotate-half RoPE, non-causal multi-head attention with grouped
 * KV heads, SwiGLU MLP, final RMSNorm, untied LM head, no biases).
 * Requirements: n_heads % n_kv_heads == 0; 0 <= mask_id < vocab.
 * DLLM_BF16: head_dim == 128, d_model % 256 == 0, d_ff % 128 == 0, n_heads and
 * n_kv_heads even.  DLLM_F32: head_dim in {64, 128}, sequence length <= 8000.
 */
typedef struct dllm_model_cfg {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, mask_id;
  float rms_eps;
  double rope_base;
  int32_t dtype; /* DLLM_F32 or DLLM_BF16 */
} dllm_model_cfg;

/* Controller switches (Section 4.6: gating ON = BUDGET | GRIND). */
enum {
  DLLM_F_BLOCK_SCHED = 1u, /* Box 4: theta_e^(b) decreases with the block index        */
  DLLM_F_POS = 2u,         /* Box 6: position factor and clip; off: theta_i = theta_b(t) */
  DLLM_F_BUDGET = 4u,      /* Box 5: per-token step budgets B_i                           */
  DLLM_F_GRIND = 8u,       /* Box 7: grinding detector and its fallback commit            */
  /* Fixed-schedule baseline (the "Fixed" column of Section 6's step-reduction
   * table) instead of the confidence-aware rule: at local step t each sequence
   * commits its floor(bl/T) masked tokens of highest confidence (one more in
   * the first bl % T steps; equal confidence: lower position first; NaN ranks
   * lowest), reason DLLM_R_FIXED.  s, budget and ell are left untouched; the
   * other switches and the threshold constants are ignored. */
  DLLM_F_FIXED = 16u
};

/*
 * Controller constants (Boxes 3-7, Section 5); defaults in brackets.
 * Schedule values are doubles: thresholds are evaluated in float64, clipped,
 * then rounded to float32; confidences are compared in float32.
 *   theta_e^(b)  = max(theta_e - theta_e_step * (b-1), theta_e_floor), b 1-based
 *   theta_b(t)   = theta_s                                 if t < warmup*T
 *                = theta_e^(b) + (theta_s - theta_e^(b))/2 * (1 + cos(pi u)),
 *                  u = (t - warmup*T) / (T - warmup*T)     otherwise
 *   theta_i(t)   = clip(theta_b(t) * pos_factor[band(p)], clip_lo, clip_hi)
 *   band(p)      = number of pos_edge[] entries <= p (in-block position p)
 *   B_i          = budget_easy if s_i > s_easy and p < p_easy; else
 *                  budget_hard if s_i < s_hard or p >= p_hard; else budget_mid
 *   commit       : c_i >= theta_i(t), or (BUDGET) t >= B_i
 *   grinding     : eta(t) < eta_bar for `patience` consecutive steps; then
 *                  masked tokens with c_i > theta_fb commit and the block ends.
 * Masked tokens left when a block ends (grinding, last step) take their
 * current argmax ("flush").  eta counts tokens; eta_bar [1.5].
 * Requirements: 1 <= block_len <= 64; 1 <= T; 0 <= warmup < 1; finite values.
 */
typedef struct dllm_cai_params {
  int32_t block_len;         /* [32]                                    */
  int32_t steps_per_block;   /* T; 0 means block_len                    */
  double theta_s;            /* [0.90] */
  double theta_e;            /* [0.70] */
  double theta_e_step;       /* [0.10] */
  double theta_e_floor;      /* [0.40] */
  double warmup;             /* [0.15] */
  int32_t pos_edge[3];       /* [16, 32, 48] */
  double pos_factor[4];      /* [0.80, 0.90, 1.05, 1.10] */
  double clip_lo, clip_hi;   /* [0.20, 0.98] */
  float s_easy, s_hard;      /* [0.50, 0.25] */
  int32_t p_easy, p_hard;    /* [32, 48] */
  int32_t budget_easy, budget_mid, budget_hard; /* [8, 32, 64] */
  double eta_bar;            /* [1.5] */
  int32_t patience;          /* K [4] */
  float theta_fb;            /* [0.40] */
  uint32_t flags;            /* DLLM_F_* */
} dllm_cai_params;

/* Reason codes stored per committed token. */
enum {
  DLLM_R_MASKED = 0,
  DLLM_R_THRESH = 1,
  DLLM_R_BUDGET = 2,
  DLLM_R_GRIND = 3,
  DLLM_R_FLUSH = 4,
  DLLM_R_FIXED = 5
};

/*
 * Decoding state: all device pointers, caller-owned, updated in place.
 * Together with (block, t) it is the complete state of Algorithm 1, so a
 * decode can be stopped after any step and resumed from a copy.
 */
typedef struct dllm_state {
  int32_t* x;           /* [B, L]  token ids; mask_id where masked                 */
  int32_t* commit_step; /* [B, G]  local step t of the commit, -1 while masked      */
  int8_t* reason;       /* [B, G]  DLLM_R_*                                         */
  float* s;             /* [B, G]  first-step confidence s_i (Box 2)                */
  int32_t* budget;      /* [B, G]  B_i (Box 5)                                      */
  int32_t* ell;         /* [B]     low-yield counter of the current block           */
  int32_t* done;        /* [B]     1 once the sequence has finished the block       */
} dllm_state;

typedef struct dllm_model dllm_model;

/*
 * Bytes of the model buffer dllm_model_create needs for cfg: the bf16 LM
 * head's tiled copy (ceil(V/256)*256*d bf16 values, rounded up to 256 bytes);
 * 0 for a DLLM_F32 model.  Errors as for dllm_model_create's shape checks.
 */
int dllm_model_buffer_size(const dllm_model_cfg* cfg, size_t* bytes);

/*
 * Create a model handle from caller-owned device weights (borrowed for the
 * handle's lifetime).  `weights` is a host array of n_weights =
 * 3 + 9*n_layers device pointers in this order, each row-major, of cfg.dtype
 * (norm gains included):
 *   embed [V, d]; per layer: attn_norm [d], wq [Hq*hd, d], wk [Hkv*hd, d],
 *   wv [Hkv*hd, d], wo [d, Hq*hd], mlp_norm [d], w_gate [F, d], w_up [F, d],
 *   w_down [d, F]; then final_norm [d], lm_head [V, d].
 * model_buf: device, 256-byte aligned, at least dllm_model_buffer_size()
 * bytes, borrowed for the handle's lifetime (may be NULL for DLLM_F32).  For
 * DLLM_BF16 a copy of lm_head in the tiled layout that the LM-head kernel
 * streams contiguously is written there, enqueued on `stream` (ordered after
 * the caller's earlier work on that stream; other streams must be ordered by
 * the caller): later writes to the caller's lm_head are not seen.  All other
 * weights are read in place on every call.
 * Errors: DLLM_EINVAL (null pointer, bad count, misaligned buffer),
 * DLLM_ENOMEM (model_buf too small), DLLM_EUNSUPPORTED (shape, or a bf16 LM
 * head above 2 GiB), DLLM_EHIP.
 */
int dllm_model_create(const dllm_model_cfg* cfg, const void* const* weights, int32_t n_weights, void* model_buf,
                      size_t model_buf_bytes, void* stream, dllm_model** out);
int dllm_model_destroy(dllm_model* model);

/*
 * Optional, bf16 models: copies of every layer's q/k/v, output, gate/up and
 * down weights in the tiled MFMA-operand order of the LM head's copy (each
 * 256-row x 64-k block one contiguous 32 KiB run) in the caller's buffer
 * `buf` (device, 256-byte aligned, at least dllm_model_packed_size() bytes:
 * about the size of those weights, ~14 GB for the LLaDA-8B shape), borrowed
 * for the handle's lifetime and enqueued on `stream` as for the model buffer.
 * GEMMs of at most 128 rows -- the block rows of a cached step
 * (dllm_forward_kv and friends) -- then stream these runs instead of the
 * row-major tensors: up to 64 rows through a register-direct kernel (k summed
 * in another order: results agree to rounding, not bit for bit), 65 .. 128
 * rows through the tiled kernel (bit-identical).  Later writes to the
 * caller's weights are not seen.  A later call repacks into its own buffer.
 * Errors: DLLM_EUNSUPPORTED (fp32 model), DLLM_EINVAL, DLLM_ENOMEM, DLLM_EHIP.
 */
int dllm_model_packed_size(const dllm_model* model, size_t* bytes);
int dllm_model_pack_weights(dllm_model* model, void* buf, size_t bytes, void* stream);

/*
 * Bytes of workspace needed by dllm_forward / dllm_step / dllm_generate for
 * B sequences of length L whose LM head runs on `rows` positions per sequence
 * (the block length for a step).
 */
int dllm_workspace_size(const dllm_model* model, int32_t B, int32_t L, int32_t rows, size_t* bytes);

/* Byte offsets of the intermediate buffers inside the workspace (for tests
 * that check each stage against a reference).  Layouts:
 *   h      float32 [B*L, d]             residual stream
 *   a_attn act     [B*L, d]             RMSNorm output feeding q/k/v
 *   q      act     [B, Hq, L, hd]       after RoPE
 *   k      act     [B, Hkv, L, hd]      after RoPE
 *   vt     act16   [B, Hkv, hd, L]      v transposed (positions contiguous)
 *   attn   act     [B*L, Hq*hd]         attention output
 *   a_mlp  act     [B*L, d]             RMSNorm output feeding the MLP
 *   u      act     [B*L, F]             silu(gate) * up
 *   hb     act     [B*rows, d]          final RMSNorm of the head rows
 * act = float32 for DLLM_F32 models, bf16 for DLLM_BF16 models; act16 =
 * float32 for DLLM_F32 models and, for DLLM_BF16 models, the bf16 values of v
 * stored as IEEE half (exact within half's range) for the attention kernel's
 * half-precision probability x value product.  Every buffer up to u, the RoPE
 * tables and the error word lie at offsets that do not depend on `rows`, so
 * calls with different row counts (dllm_layer, then dllm_head) can share one
 * workspace of the largest size. */
typedef struct dllm_ws_layout {
  size_t total, h, a_attn, q, k, vt, attn, a_mlp, u, hb;
} dllm_ws_layout;
int dllm_workspace_layout(const dllm_model* model, int32_t B, int32_t L, int32_t rows, dllm_ws_layout* out);

/* h[b*L + l, :] = embed[x[b, l], :] as float32 into the workspace's h.
 * x: device int32 [B, L], each in [0, vocab).  An id outside that range is
 * never used as an address: its row of h is zero and the workspace's error
 * word records it (reported by the next commit on this workspace: see
 * dllm_step). */
int dllm_embed(const dllm_model* model, const int32_t* x, int32_t B, int32_t L, void* workspace,
               size_t workspace_bytes, void* stream);

/* One transformer layer (0 <= layer < n_layers) on the workspace's h, in place.
 * part = 0: attention half (norm, q/k/v + RoPE, attention, output projection
 * + residual); part = 1: MLP half (norm, SwiGLU, down projection + residual);
 * part = 2: both. */
int dllm_layer(const dllm_model* model, int32_t layer, int32_t part, int32_t B, int32_t L, void* workspace,
               size_t workspace_bytes, void* stream);

/*
 * Final RMSNorm and LM head on rows [row0, row0 + rows) of every sequence of
 * the workspace's h, fused with the vocabulary reduction of Box 1:
 *   conf[b*rows + r]   = max_v softmax(logits)_v over v != mask_id   (float32)
 *   argmax[b*rows + r] = lowest v != mask_id with the largest logit (int32)
 * logits: optional device float32 [B*rows, V] (NULL on the hot path; when set
 * the logits are also written out, mask_id column included, unmasked).
 */
int dllm_head(const dllm_model* model, int32_t B, int32_t L, int32_t row0, int32_t rows, float* conf,
              int32_t* argmax, float* logits, void* workspace, size_t workspace_bytes, void* stream);

/*
 * dllm_head without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same final RMSNorm + LM head + vocabulary reduction,
 * with the same kernels and results bit for bit, reading the final residual
 * from the caller's h (device float32 [B*L, d], 16-byte aligned, read only)
 * and keeping its scratch (normed rows, per-workgroup partials, the merge
 * ticket) in a static device array of 8 MiB that the library holds on each GPU
 * it runs on until the process ends.  No call allocates.  The array is shared
 * by every call on that GPU: calls that overlap on one GPU (other streams,
 * other threads) race and must be ordered by the caller; each call starts by
 * zeroing what must start at zero.  conf/argmax/logits as for dllm_head.
 * Errors: DLLM_ENOMEM when the head rows need more than the static scratch
 * (bf16: up to 256 rows at d <= 8192 fit; float32: B*rows*(d + V)*4 bytes
 * must fit), the checks of dllm_head otherwise.
 */
int dllm_head_noalloc(const dllm_model* model, const float* h, int32_t B, int32_t L, int32_t row0, int32_t rows,
                      float* conf, int32_t* argmax, float* logits, void* stream);

/* dllm_embed + every layer + dllm_head: one forward on x [B, L] (device).
 * Afterwards the workspace's h holds the final residual of the head rows only
 * (the last layer's split-K partials are added by the final norm to those
 * rows alone). */
int dllm_forward(const dllm_model* model, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                 float* conf, int32_t* argmax, float* logits, void* workspace, size_t workspace_bytes,
                 void* stream);

/*
 * Initialise `state` for a decode: x = [prompt | mask_id * G], commit_step =
 * -1, reason = 0, s = 0, budget = 0, ell = 0, done = 0.  prompt: device int32
 * [B, P], each in [0, vocab) and != mask_id.
 */
int dllm_state_init(int32_t mask_id, const int32_t* prompt, int32_t B, int32_t P, int32_t G, dllm_state* state,
                    void* stream);

/*
 * The controller for one step (Algorithm 1's body) of block `block` (0-based)
 * at local step t, from this step's predictions conf/argmax (device, [B, bl],
 * position p of the block at index b*bl + p).  At t = 0 it first resets ell and
 * done and stores s and B_i.  Sequences whose done flag is set are left
 * unchanged.  all_done (device int32, optional) receives 1 when every
 * sequence has finished the block.  mask_id is the model's mask token.
 */
int dllm_commit(const dllm_cai_params* params, dllm_state* state, const float* conf, const int32_t* argmax,
                int32_t B, int32_t P, int32_t G, int32_t block, int32_t t, int32_t mask_id, int32_t* all_done,
                void* stream);

/*
 * One denoising step: dllm_forward on state->x for block `block`'s rows, then
 * dllm_commit.  conf_out / argmax_out: optional device [B, bl] copies of the
 * step's predictions (NULL on the hot path).  all_done_host: optional host
 * int32; when given the call waits for the step (polling the word the commit
 * kernel publishes to the model's pinned flag) and stores 1 there when
 * every sequence has finished the block, and reports the workspace's error
 * word (then cleared): DLLM_EINVAL if a token id of x was outside [0, vocab)
 * (its embedding was taken as zero), DLLM_EUNSUPPORTED if a value of v was
 * beyond IEEE half's range (the attention's half-precision P.V operand; it
 * was used as +-65504).  The step's decisions were still applied.
 */
int dllm_step(const dllm_model* model, const dllm_cai_params* params, dllm_state* state, int32_t B, int32_t P,
              int32_t G, int32_t block, int32_t t, float* conf_out, int32_t* argmax_out, int32_t* all_done_host,
              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decode G tokens after the prompt (device int32 [B, P]), block by block
 * (Section 4.3), running dllm_step until each block finishes.  Waits for the
 * stream once per step (the block-finished flag) and returns after the last
 * step, or after the first step whose error word is set (the errors of
 * dllm_step).  The RoPE tables are built once, before the first step.
 * forwards_host: optional host int32 [G/bl], forwards run per block.
 * conf_trace / argmax_trace: optional device [G/bl, T, B, bl] records of every
 * step's predictions (entries of steps not run are left untouched).
 * total_forwards: optional host int32.
 */
int dllm_generate(const dllm_model* model, const dllm_cai_params* params, const int32_t* prompt, int32_t B,
                  int32_t P, int32_t G, dllm_state* state, int32_t* forwards_host, int32_t* total_forwards,
                  float* conf_trace, int32_t* argmax_trace, void* workspace, size_t workspace_bytes,
                  void* stream);

/*
 * Cross-step key/value reuse (Section 5: the decoder runs on a KV cache
 * refreshed every 16 steps for LLaDA and 8 for Dream; the paper does not
 * define the cache further).  Reading implemented: local step t of a block is
 * a refresh step when t % refresh_every == 0; a refresh step runs the full
 * forward and stores every layer's keys (after RoPE) and values for all L
 * positions; any other step runs only the current block's rows through the
 * layers, attending over the stored keys/values of the other positions (as of
 * the last refresh) and the block rows' fresh ones, which are written into the
 * cache at the block positions.  An approximation for two or more layers.
 *
 * The cache is caller-owned device memory (256-byte aligned) of
 * dllm_kv_cache_size() bytes for B sequences of L positions: per layer, keys
 * [B, Hkv, L, hd] then values transposed [B, Hkv, hd, L] (float32 for a
 * DLLM_F32 model; bf16 keys and IEEE-half values holding bf16 values for
 * DLLM_BF16), each rounded up to 256 bytes.  Calls that use it need the same
 * B and L.  Errors as for the calls above, plus DLLM_ENOMEM for a cache that
 * is too small.
 */
int dllm_kv_cache_size(const dllm_model* model, int32_t B, int32_t L, size_t* bytes);

/* refresh != 0: dllm_forward that also stores every layer's keys/values for
 * all L positions into kv_cache.  refresh == 0: the forward of rows [row0,
 * row0 + rows) of every sequence only, against the cache (conf/argmax/logits
 * of those rows as for dllm_forward).  The workspace is the one for (B, L,
 * rows). */
int dllm_forward_kv(const dllm_model* model, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                    int32_t refresh, float* conf, int32_t* argmax, float* logits, void* kv_cache, size_t kv_bytes,
                    void* workspace, size_t workspace_bytes, void* stream);

/* Stages of the cached forward, for tests: dllm_embed_rows puts the embeddings
 * of x[b, row0 + i] at the workspace's h[b*rows + i]; dllm_layer_kv runs one
 * layer (part as for dllm_layer) on those B*rows rows, writing their
 * keys/values into the layer's cache entries at positions row0 .. row0+rows-1
 * and attending over all L cached positions (rows == L, row0 == 0: the full
 * layer, filling the cache).  Workspace for (B, L, rows), or (B, L, 0) when
 * rows == L. */
int dllm_embed_rows(const dllm_model* model, const int32_t* x, int32_t B, int32_t L, int32_t row0, int32_t rows,
                    void* workspace, size_t workspace_bytes, void* stream);
int dllm_layer_kv(const dllm_model* model, int32_t layer, int32_t part, int32_t B, int32_t L, int32_t row0,
                  int32_t rows, void* kv_cache, size_t kv_bytes, void* workspace, size_t workspace_bytes,
                  void* stream);

/* dllm_step with the cache: refresh != 0 runs the full forward and refreshes
 * the cache, refresh == 0 the cached forward of the block rows. */
int dllm_step_kv(const dllm_model* model, const dllm_cai_params* params, int32_t refresh, dllm_state* state,
                 int32_t B, int32_t P, int32_t G, int32_t block, int32_t t, float* conf_out, int32_t* argmax_out,
                 int32_t* all_done_host, void* kv_cache, size_t kv_bytes, void* workspace, size_t workspace_bytes,
                 void* stream);

/* dllm_generate with cross-step key/value reuse: step t of each block
 * refreshes the cache when t % refresh_every == 0 (>= 1; 1 = every step, the
 * same decisions as dllm_generate), else runs the cached forward. */
int dllm_generate_kv(const dllm_model* model, const dllm_cai_params* params, int32_t refresh_every,
                     const int32_t* prompt, int32_t B, int32_t P, int32_t G, dllm_state* state,
                     int32_t* forwards_host, int32_t* total_forwards, float* conf_trace, int32_t* argmax_trace,
                     void* kv_cache, size_t kv_bytes, void* workspace, size_t workspace_bytes, void* stream);

/* Per-kernel timing with HIP events recorded on the launch stream around each
 * launch of the selected kernel classes.  kind: 0 = q/k/v GEMM (with RoPE),
 * 1 = attention, 2 = LM head + reduction, 3 = commit, 4 = norms and
 * embedding (with the residual GEMMs' split-K partials they fold in), 5 =
 * gate/up GEMM (with SwiGLU), 6 = output projection, 7 = down projection.
 * dllm_prof_enable(model, mask) starts recording
 * the kinds whose bit (1 << kind) is set and clears earlier records (mask 0
 * stops); dllm_prof_read waits for the recorded work and returns the summed
 * duration in milliseconds and the launch count of one kind.  Events are host
 * objects kept by the model handle (no device memory). */
int dllm_prof_enable(dllm_model* model, int32_t enable);
int dllm_prof_read(dllm_model* model, int32_t kind, double* total_ms, int64_t* launches);
/* Record only one launch in `every` (>= 1; default 1) of each enabled kind,
 * the first of each run of `every`: each record brackets its launch with two
 * events on the stream, which cost the stream a few microseconds each, so a
 * timed decode samples (e.g. one of a forward's n_layers launches of a
 * kind).  Resets the per-kind launch counts; DLLM_EINVAL if every < 1. */
int dllm_prof_every(dllm_model* model, int32_t every);

/* Message of the last failure on the calling thread ("" if none). */
const char* dllm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DLLM_H */
