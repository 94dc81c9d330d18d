/*
 * aj.h -- C ABI of libaj: the merged actor update on one MI355X (gfx950).
 *
 * The actor (policy) update over multi-turn agent trajectories, in three
 * stages:
 *   1. timeline merging          (Section 4.4.2, Algorithm 1, token- or text-level Match)
 *   2. one packed variable-length causal decoder block, forward and backward
 *   3. the fused LM head: vocab projection, log-softmax, token log-prob and the
 *      clipped policy-gradient loss (Section 3: GRPO-style updates), forward
 *      and backward, over the loss-masked tokens only.
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless marked host.  The caller allocates
 *     every buffer, including workspaces sized by the *_bytes queries; the
 *     library allocates no device memory, keeps no pointer after returning
 *     and holds no state besides a thread-local error string.
 *   - `stream` is a hipStream_t (NULL = the null stream).  All work is
 *     enqueued on it; no call synchronises the host except aj_read_device_error.
 *   - Return value: AJ_OK, or an aj_status code after which nothing was
 *     enqueued (argument errors are found on the host before any launch);
 *     aj_last_error() then describes it.  AJ_ERR_HIP means a launch failed.
 *   - Data errors that only the device can see (a token id >= vocab, a
 *     timeline whose first token does not start a block, an author value of 3)
 *     set bits in a device int32 `err` word when one is passed; the kernels
 *     then skip the bad element and finish normally.
 *   - Floating point gradients are ACCUMULATED (+=) into float32 buffers, so
 *     packs can be looped; the caller zeroes them first.
 *   - dtype AJ_F32 stores weights and activations as float32, AJ_BF16 as
 *     bfloat16 (round to nearest even); accumulation is float32 either way.
 *   - Matrices are row-major; a weight of shape [out, in] maps x[in] to y[out].
 */
#ifndef AJ_H
#define AJ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AJ_OK = 0,
  AJ_ERR_NULL = 1,          /* a required pointer is NULL */
  AJ_ERR_SHAPE = 2,         /* a size or offset is out of range / not monotone */
  AJ_ERR_UNSUPPORTED = 3,   /* a valid request the library does not implement */
  AJ_ERR_WORKSPACE = 4,     /* workspace smaller than the *_bytes query asked for */
  AJ_ERR_HIP = 5            /* a HIP launch or runtime call failed */
} aj_status;

typedef enum { AJ_F32 = 0, AJ_BF16 = 1 } aj_dtype;

/* Per-token flag byte of the unmerged timelines. */
enum {
  AJ_AUTHOR_USER = 0, AJ_AUTHOR_ENV = 1, AJ_AUTHOR_LLM = 2, AJ_AUTHOR_MASK = 3,
  AJ_FLAG_BLOCK_START = 4   /* set on the first token of every message block */
};

/* Bits of the device error word. */
enum {
  AJ_DEVERR_TOKEN_RANGE = 1,   /* a token id outside [0, vocab) */
  AJ_DEVERR_BAD_FLAGS = 2,     /* author 3, or a timeline not starting a block */
  AJ_DEVERR_EMPTY = 4,         /* an empty timeline */
  AJ_DEVERR_OFFSETS = 8,       /* offsets not monotone, out of range, or not tiling [0, n) */
  AJ_DEVERR_BLOCKS = 16        /* text-level merge: the block-start bits do not give n_blk
                                  blocks, or a timeline does not start a block */
};

const char *aj_status_str(int status);
/* Detail of the last non-OK return on this thread ("" if none). */
const char *aj_last_error(void);
/* Waits for `stream`, then copies the device error word to *host_err. */
int aj_read_device_error(const int32_t *err, void *stream, int32_t *host_err);

/* ------------------------------------------------------------------ 1. merge
 * Section 4.4.2: each intercepted LLM call yields one timeline, an ordered list
 * of message blocks (token ids, author in {user, env, llm}, per-token log-prob,
 * loss mask = 1 exactly on llm tokens).  Algorithm 1 visits timelines from the
 * last one down; each one not yet absorbed absorbs every earlier, not yet
 * absorbed timeline whose blocks it matches one by one (|T_i| >= |T_j| and
 * Match on blocks 1..|T_j|), and takes over llm authorship -- author, tokens,
 * log-prob and, here, the advantage -- on the aligned blocks where its own
 * block is not llm.  Survivors are returned in original order.
 *
 * Match here is token-level: equal token ids AND equal block boundaries
 * (block starts are the AJ_FLAG_BLOCK_START bits; blocks are never empty).
 * Authors are not compared.  Merging stays inside one episode.
 */
typedef struct {
  int32_t n_traj;               /* episodes */
  int32_t n_tl;                 /* timelines (one per LLM call), all episodes */
  int64_t n_tok;                /* unmerged tokens, < 2^31 */
  const int32_t *traj_tl_off;   /* [n_traj+1] timelines of episode e: [off[e], off[e+1]), collection order */
  const int64_t *tl_tok_off;    /* [n_tl+1]   tokens of timeline i: [off[i], off[i+1]) */
  const int32_t *tok;           /* [n_tok] token ids */
  const uint8_t *flags;         /* [n_tok] author | AJ_FLAG_BLOCK_START */
  const float *old_logprob;     /* [n_tok] rollout log-prob; read where author == llm */
  const float *adv;             /* [n_tok] advantage; read where author == llm */
} aj_timelines;

typedef struct {
  /* per timeline / segment; capacity n_tl (+1) */
  int32_t *absorber;            /* [n_tl] -1 = survivor, else global index of the absorbing timeline */
  int32_t *cu_seqlens;          /* [n_tl+1] segment token offsets; entries past n_seg are left alone */
  int32_t *seg_src;             /* [n_tl]   timeline each segment comes from */
  int32_t *cu_targets;          /* [n_tl+1] offsets of each segment's masked targets in `targets` */
  int64_t *counts;              /* [4] n_seg, n_tok_out, n_mask (= number of targets), max_seqlen */
  /* per output token; capacity n_tok (merged output is never longer than the input) */
  int32_t *tok;
  int32_t *pos;                 /* position inside its segment, from 0 */
  uint8_t *mask;                /* 1 on llm tokens after the transfers */
  float *old_logprob;           /* the llm token's rollout log-prob, 0 elsewhere */
  float *adv;                   /* the llm token's advantage, 0 elsewhere */
  int32_t *targets;             /* [n_tok] ascending output positions p with mask[p] == 1 that do
                                   not start a segment: the tokens the loss scores */
} aj_packed;

/* Workspace for aj_merge_timelines / aj_flatten_timelines. */
size_t aj_merge_workspace_bytes(int32_t n_traj, int32_t n_tl, int64_t n_tok);
/* Algorithm 1 over every episode, then the survivors laid end to end.
 * The offsets must tile [0, n_tok) and [0, n_tl) exactly (else
 * AJ_DEVERR_OFFSETS, and every count comes back 0).  Result is independent of
 * the launch: bit-identical on every call. */
int aj_merge_timelines(const aj_timelines *in, aj_packed *out, int32_t *err,
                       void *ws, size_t ws_bytes, void *stream);
/* The same outputs without merging: every timeline is its own segment
 * (absorber all -1).  The unmerged baseline the paper compares against. */
int aj_flatten_timelines(const aj_timelines *in, aj_packed *out, int32_t *err,
                         void *ws, size_t ws_bytes, void *stream);

/* aj_merge_timelines for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  It takes no workspace argument; its workspace is a built-in
 * device array of aj_merge_noalloc_max_workspace_bytes() bytes (64 MiB), one
 * per GPU, held until the process ends and reused by every call on that GPU.
 * Inputs whose aj_merge_workspace_bytes exceeds it are refused with
 * AJ_ERR_WORKSPACE before anything is enqueued (about 470M unmerged tokens in
 * few timelines; each timeline also takes ~60 bytes).
 * Outputs, errors and results are those of aj_merge_timelines, bit for bit.
 * The call allocates nothing (no hipMalloc or hipFree); the first call on a
 * device looks up that device's copy of the array.  Calls that overlap on
 * one GPU (several streams or threads at once) share the array and race:
 * serialise them. */
size_t aj_merge_noalloc_max_workspace_bytes(void);
int aj_merge_timelines_noalloc(const aj_timelines *in, aj_packed *out, int32_t *err,
                               void *stream);

/* ------------------------------------------------------------------ 1b. merge, text-level Match
 * Section 4.4.2, Relaxed Matching Strategies: Match compares the MESSAGE TEXT
 * of aligned blocks instead of their token ids (the paper's default
 * strategy).  It tolerates tokenizer drift: a chat template that re-renders an
 * earlier message differently (for instance without its thinking section)
 * keeps the text and changes the ids, so token-level Match would keep the two
 * timelines apart.  The library never sees text: the caller passes one 64-bit
 * key per block, with equal text <=> equal key (an interned message id is
 * exact; a 64-bit hash of the text is exact up to collisions).
 *
 * A transfer copies the absorbed block's tokens, log-probs and advantages
 * over the survivor's block (Algorithm 1), so a block -- and its segment --
 * can change length; the output is laid out again from the chosen blocks
 * (every input block lands in at most one place, so the output is still never
 * longer than the input).  A block's author is the author bits of its first
 * token; mask is 1 on every token of an llm block of the output.
 *
 * Train-inference (TI) consistency report, `ti` [2] (optional, int64): the
 * llm blocks of the output -- and their tokens -- whose tokens before them in
 * their output segment differ from the tokens before them in the timeline
 * that generated them: log-probs the update scores in a context other than
 * the one they were sampled in.  Token-level Match never produces any.
 */
typedef struct {
  int32_t n_blk;                /* blocks of all timelines = number of AJ_FLAG_BLOCK_START bits */
  const uint64_t *key;          /* [n_blk] text key of each block, blocks in token order */
} aj_block_texts;

/* Workspace for aj_merge_timelines_text. */
size_t aj_merge_text_workspace_bytes(int32_t n_traj, int32_t n_tl, int64_t n_tok, int32_t n_blk);
/* Algorithm 1 with text-level Match; outputs as aj_merge_timelines.  Beyond
 * its device errors, block-start bits that do not give n_blk blocks, or a
 * timeline that does not start a block, raise AJ_DEVERR_BLOCKS and every
 * count comes back 0.  `ti` may be NULL.  Bit-identical on every call. */
int aj_merge_timelines_text(const aj_timelines *in, const aj_block_texts *text, aj_packed *out,
                            int64_t *ti, int32_t *err, void *ws, size_t ws_bytes, void *stream);

/* Host: greedy in-order packing of segments into packs of at most max_tokens
 * tokens (a longer segment gets a pack of its own).  cu_seqlens is a HOST copy
 * [n_seg+1]; pack_seg_off (HOST, capacity n_seg+1) receives the first segment
 * of each pack plus a final n_seg; *n_packs receives the pack count. */
int aj_plan_packs(const int32_t *cu_seqlens, int32_t n_seg, int32_t max_tokens,
                  int32_t *pack_seg_off, int32_t *n_packs);

/* ------------------------------------------------------------------ embedding
 * The first layer of the policy that scores each sample's tokens (Section 3:
 * a sample is a token sequence used for policy optimization; Section 4.2,
 * step (4): the update trains the full model weights, the embedding
 * included).  The policy's architecture is not given by the paper; the
 * embedding is the input table of the decoder models it trains (Section 5).
 */
/* x[p] = emb[tok[p]] for p < n_tok; emb [vocab, d], x [n_tok, d] in `dtype`.
 * A token outside [0, vocab) gives a zero row and sets AJ_DEVERR_TOKEN_RANGE
 * in *err (err may be NULL). */
int aj_embed_fwd(const int32_t *tok, int32_t n_tok, const void *emb, int32_t d, int32_t vocab,
                 int dtype, void *x, int32_t *err, void *stream);
/* Workspace bytes of aj_embed_bwd for n_tok rows of width d. */
size_t aj_embed_bwd_workspace_bytes(int32_t n_tok, int32_t d);
/* The embedding gradient: d_emb[v] += sum of dx[p] over the positions p with
 * tok[p] == v (float32; d_emb [vocab, d], dx [n_tok, d], both 16-byte
 * aligned, d a multiple of 4, n_tok <= 2^30).  Deterministic: each row of
 * d_emb receives one addition, the rows of its token summed in ascending
 * position order (no float atomics), so the result is bit-identical on
 * every call.  Tokens outside [0, vocab) contribute nothing.  ws: at least
 * aj_embed_bwd_workspace_bytes(n_tok, d) bytes, else AJ_ERR_WORKSPACE. */
int aj_embed_bwd(const int32_t *tok, int32_t n_tok, const float *dx, int32_t d, int32_t vocab,
                 float *d_emb, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------ 2. block
 * The policy's forward and backward over the merged samples: Section 4.4.2
 * (Timeline Merging) merges timelines precisely so that the actor update
 * does not run the shared prefix of every call again -- each surviving
 * timeline is one segment, attended causally within itself only -- and
 * Section 4.2, step (4) then computes the policy-gradient loss and updates
 * the weights.  The paper trains Qwen-family decoders (Section 5) and gives
 * no architecture; the block below is that standard decoder layer.
 * One pre-norm decoder block over a pack of segments laid end to end:
 *   a = RMSNorm(x)*g1; q,k,v = a W_qkv^T; rotate-half RoPE on q,k at `pos`
 *   (inverse frequency theta^(-2i/head_dim)); o = causal softmax(q k^T/sqrt(hd)) v
 *   inside each segment, query head h reading kv head floor(h*Hkv/Hq);
 *   x1 = x + o W_o^T; b = RMSNorm(x1)*g2;
 *   y = x1 + (silu(b W_gate^T) * b W_up^T) W_down^T.
 * W_qkv rows: Hq*hd query rows, then Hkv*hd key rows, then Hkv*hd value rows.
 * W_gate_up rows: d_ff gate rows, then d_ff up rows.
 */
typedef struct {
  int32_t d_model, n_q_heads, n_kv_heads, head_dim, d_ff;
  float rms_eps;
  float rope_theta;
  int32_t dtype;                /* aj_dtype of weights, x, y and saved activations */
} aj_block_cfg;

typedef struct {
  const void *attn_norm;        /* [d] */
  const void *w_qkv;            /* [(Hq+2Hkv)*hd, d] */
  const void *w_o;              /* [d, Hq*hd] */
  const void *mlp_norm;         /* [d] */
  const void *w_gate_up;        /* [2*d_ff, d] */
  const void *w_down;           /* [d, d_ff] */
  /* Optional, bfloat16 only: the same four projection weights stored
   * transposed, [in][out] -- all four or none (NULL).  When given, the
   * forward's projections read these: their rows reach the matrix cores
   * faster than those of the [out][in] copies (3-6 % on the 32B-class
   * shapes).  The caller keeps them equal to the weights above
   * (aj_transpose_bf16 after every update); the backward, the float32 path
   * and the LoRA stack read only the weights above. */
  const void *w_qkv_t;          /* [d, (Hq+2Hkv)*hd] */
  const void *w_o_t;            /* [Hq*hd, d] */
  const void *w_gate_up_t;      /* [d, 2*d_ff] */
  const void *w_down_t;         /* [d_ff, d] */
} aj_block_weights;

typedef struct {                /* float32, accumulated */
  float *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
} aj_block_grads;

typedef struct {
  int32_t n_tok;                /* tokens in the pack */
  int32_t n_seg;                /* segments in the pack */
  int32_t max_seqlen;           /* longest segment (host value) */
  int32_t base;                 /* cu_seqlens values are offsets + base (a slice of a
                                   batch-wide array): row r of the pack is offset r + base */
  const int32_t *cu_seqlens;    /* [n_seg+1], cu_seqlens[0] == base, cu_seqlens[n_seg] == base + n_tok */
  const int32_t *pos;           /* [n_tok] position of each token inside its segment (RoPE) */
} aj_varlen;

/* Bytes of the activation arena the forward fills and the backward reads. */
size_t aj_block_saved_bytes(const aj_block_cfg *cfg, int32_t n_tok);
/* Scratch for either direction. */
size_t aj_block_workspace_bytes(const aj_block_cfg *cfg, int32_t n_tok, int32_t n_seg);
/* x, y: [n_tok, d] in cfg->dtype.  `saved` (aj_block_saved_bytes) receives
 * the activations the backward reads and must outlive it; ws: at least
 * aj_block_workspace_bytes bytes.  Errors: AJ_ERR_NULL for a missing
 * pointer, AJ_ERR_SHAPE for sizes or offsets out of range or query heads
 * that do not group evenly over the key/value heads, AJ_ERR_UNSUPPORTED for
 * a head_dim outside 8..128 (multiple of 8) or another dtype,
 * AJ_ERR_WORKSPACE for a short workspace. */
int aj_varlen_block_fwd(const aj_block_cfg *cfg, const aj_block_weights *w, const aj_varlen *vl,
                        const void *x, void *y, void *saved, void *ws, size_t ws_bytes,
                        void *stream);
/* The gradient of the block: dy, dx float32 [n_tok, d] (dx is written, not
 * accumulated; dx may alias dy); every weight gradient in g is float32 and
 * accumulated (+=), summed over tokens in a fixed order (bit-identical on
 * every call).  x and `saved` must be the forward's.  Errors as the
 * forward. */
int aj_varlen_block_bwd(const aj_block_cfg *cfg, const aj_block_weights *w, const aj_varlen *vl,
                        const void *x, const void *saved, const float *dy, float *dx,
                        const aj_block_grads *g, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------ 2b. layer stack
 * A policy of n_layers such blocks, each with its own weights, the output of
 * one the input of the next (step (4) of Section 4.2 updates the whole model;
 * the stack is the standard decoder).  Activation checkpointing: the forward
 * keeps each layer's INPUT -- x for layer 0, then n_layers-1 slabs of
 * [n_tok, d] in `ckpt` -- and leaves the last layer's saved activations in
 * `saved`.  The backward runs the last layer's backward, then for each earlier
 * layer recomputes its forward into the same `saved` arena (rewriting its
 * output slab with the same values) right before its backward.  Memory: one
 * arena plus (n_layers-1)*n_tok*d elements instead of n_layers arenas; cost:
 * one more forward of every layer but the last.  With n_layers == 1 these
 * are aj_varlen_block_fwd / _bwd and ckpt may be NULL.
 * w, g: HOST arrays of n_layers structs holding device pointers.
 * x must stay unchanged from the forward to the backward and alias nothing;
 * dx may alias dy; `saved` and `ckpt` must not be touched in between.
 */
size_t aj_stack_ckpt_bytes(const aj_block_cfg *cfg, int32_t n_layers, int32_t n_tok);
int aj_stack_fwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                 const aj_varlen *vl, const void *x, void *y, void *ckpt, void *saved,
                 void *stream);
/* ws: aj_block_workspace_bytes(cfg, n_tok, n_seg). */
int aj_stack_bwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                 const aj_varlen *vl, const void *x, void *ckpt, void *saved, const float *dy,
                 float *dx, const aj_block_grads *g, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------ 2c. LoRA
 * Section 4.2, step (4): the update may train LoRA matrices (Hu et al.)
 * instead of the full weights.  Each of the four projections of every block,
 * with frozen weight W [out, in], becomes
 *   P(v) = v W^T + scale * (v A^T) B^T,     A [rank, in], B [out, rank]
 * (qkv: in d, out (Hq+2Hkv)*hd, before RoPE; o: in Hq*hd, out d; gate_up: in
 * d, out 2*d_ff; down: in d_ff, out d).  Only A and B train: the block's
 * weights and norm gains get no gradient (and the caller leaves the embedding
 * and the LM head frozen too: aj_logprob_pg_loss_bwd takes NULL for their
 * gradients).  A, B are row-major in cfg->dtype; the products v A^T and
 * d_out B are scaled and rounded once to cfg->dtype.  rank: a multiple of 8,
 * 8..256, the same (with the same scale) in every layer.
 * The forward and backward are those of the layer stack (2b), checkpointed
 * the same way; `saved` holds aj_lora_saved_bytes (the block's activations
 * plus the four v A^T products), the backward workspace is
 * aj_lora_workspace_bytes.  lora, g: HOST arrays of n_layers structs.
 */
typedef struct {
  int32_t rank;
  float scale;                  /* alpha / rank */
  const void *a_qkv, *b_qkv, *a_o, *b_o, *a_gate_up, *b_gate_up, *a_down, *b_down;
} aj_lora;

typedef struct {                /* float32, accumulated */
  float *a_qkv, *b_qkv, *a_o, *b_o, *a_gate_up, *b_gate_up, *a_down, *b_down;
} aj_lora_grads;

size_t aj_lora_saved_bytes(const aj_block_cfg *cfg, int32_t rank, int32_t n_tok);
size_t aj_lora_workspace_bytes(const aj_block_cfg *cfg, int32_t rank, int32_t n_tok);
int aj_stack_lora_fwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                      const aj_lora *lora, const aj_varlen *vl, const void *x, void *y,
                      void *ckpt, void *saved, void *stream);
int aj_stack_lora_bwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                      const aj_lora *lora, const aj_varlen *vl, const void *x, void *ckpt,
                      void *saved, const float *dy, float *dx, const aj_lora_grads *g, void *ws,
                      size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------ 3. loss
 * The final norm, the vocab projection, the token log-prob and the clipped
 * policy-gradient objective of the actor update (Section 3, the GRPO/PPO-style
 * update the agents are trained with; the merged timelines of Section 4.4.2
 * are scored through it unchanged).
 * hn = RMSNorm(h) * g_final; for every target position p (targets[i]):
 *   logprob[i] = log softmax(hn[p-1] W_vocab^T)[tok[p]]
 *   r = exp(logprob[i] - old_logprob[p])
 *   loss += -min(r A, clip(r, 1-eps, 1+eps) A) * inv_n_mask,   A = adv[p]
 * The vocab projection is streamed: logits never reach memory in the forward
 * (unless cfg->keep_logits asks for them); the backward forms d logits one
 * vocab_chunk-wide slab per launch and keeps at most two slabs (bfloat16
 * chunks of up to 16384 columns, paired so that the d hidden and d W_vocab
 * products run once per pair; otherwise one).
 * d loss / d logprob = -A r inv_n_mask where the unclipped branch is active
 * ((A > 0 and r <= 1+eps) or (A < 0 and r >= 1-eps)), else 0.
 * Optional KL penalty against a reference policy (the low-variance KL the
 * GRPO recipe of Section 6 names, coefficient kl_coef): with
 * delta = ref_logprob[i] - logprob[i],
 *   kl = exp(delta) - delta - 1, clamped to [-10, 10],
 *   loss += kl_coef * kl * inv_n_mask,  d loss / d logprob += kl_coef * (1 - exp(delta)) * inv_n_mask
 * (the clamped side contributes no gradient).
 * Only the rows feeding a target are touched: the loss does not depend on
 * the logits of any other row.
 */
typedef struct {
  int32_t d_model, vocab, vocab_chunk;
  float clip_eps;
  float rms_eps;
  int32_t dtype;                /* aj_dtype of h, final_norm, w_vocab */
  int32_t keep_logits;          /* bfloat16 only: 1 = the forward also writes the float32
                                   logits of every scored row into `saved` (n_tgt x vocab
                                   floats, counted by aj_loss_saved_bytes) and the backward
                                   reads them instead of recomputing the vocab projection;
                                   the results are bitwise those of the recomputing
                                   backward.  0 = recompute (saved holds only hn, rstd). */
} aj_loss_cfg;

typedef struct {
  int32_t n_tok;                /* rows of h (one pack) */
  int32_t n_tgt;                /* targets scored in this call */
  int32_t row_base;             /* h row of position p is p - row_base */
  const int32_t *targets;       /* [n_tgt] positions p, row_base < p < row_base + n_tok + 1,
                                   each scored from h row p - 1 - row_base */
  const int32_t *tok;           /* token ids, indexed by p */
  const float *old_logprob;     /* indexed by p */
  const float *adv;             /* indexed by p */
  float inv_n_mask;             /* 1 / (loss-masked tokens of the WHOLE batch) */
  const float *ref_logprob;     /* [n_tgt] reference-policy log-prob of each target, or NULL */
  float kl_coef;                /* KL penalty weight; no KL term when 0 or ref_logprob NULL */
  const void *w_vocab_t;        /* optional: w_vocab transposed, [d, vocab], equal to
                                   w_vocab (vocab a multiple of 8, else AJ_ERR_SHAPE); the
                                   bfloat16 vocab projections of the forward and of the
                                   backward's recompute then read it (faster rows, as for
                                   aj_block_weights); the float32 path ignores it.  NULL =
                                   w_vocab only */
} aj_loss_in;

size_t aj_loss_saved_bytes(const aj_loss_cfg *cfg, int32_t n_tgt);
size_t aj_loss_workspace_bytes(const aj_loss_cfg *cfg, int32_t n_tgt);
/* h [n_tok, d], final_norm [d], w_vocab [vocab, d] in cfg->dtype.
 * logprob, lse: [n_tgt] float32 (written).  stats: float32[5] accumulated:
 * [0] loss (policy-gradient plus KL terms, already scaled by inv_n_mask),
 * [1] clipped-branch count, [2] sum of r, [3] targets seen, [4] sum of kl
 * (unscaled; 0 without the KL term).  `saved` (aj_loss_saved_bytes) keeps the
 * normalised rows for the backward. */
int aj_logprob_pg_loss_fwd(const aj_loss_cfg *cfg, const aj_loss_in *in, const void *h,
                           const void *final_norm, const void *w_vocab, void *saved,
                           float *logprob, float *lse, float *stats, int32_t *err,
                           void *ws, size_t ws_bytes, void *stream);
/* dh: float32 [n_tok, d], WRITTEN (rows that feed no target become 0).
 * `saved` must come from the forward of the same call (same cfg, in, h,
 * weights): with keep_logits it holds that forward's logits. 
 * d_final_norm [d], d_w_vocab [vocab, d]: float32, accumulated; NULL = that
 * weight is frozen and its gradient is not computed. */
int aj_logprob_pg_loss_bwd(const aj_loss_cfg *cfg, const aj_loss_in *in, const void *h,
                           const void *final_norm, const void *w_vocab, const void *saved,
                           const float *logprob, const float *lse, float *dh,
                           float *d_final_norm, float *d_w_vocab, void *ws, size_t ws_bytes,
                           void *stream);

/* ------------------------------------------------------------------ 4. around the update
 * GRPO advantages (Section 3: GRPO-style updates; groups of rollouts per
 * task, e.g. group size 8 in Section 5.3).  The episodes of group g are
 * [group_off[g], group_off[g+1]) (group_off: [n_groups+1], tiling the
 * episodes in order).  With the group's mean mu and sample standard deviation
 * sd (Bessel's correction):
 *   ep_adv[e] = (reward[e] - mu) / (sd + eps)
 * Section 4.3's strategy C3 trains only on groups whose rewards are not all
 * equal: ep_keep[e] = 1 iff e's group holds two different rewards; otherwise
 * (one distinct reward, or a group of one) ep_adv[e] = 0 and ep_keep[e] = 0.
 * float32 arithmetic; the keep decision compares rewards exactly.  Offsets
 * that are not monotone from 0 raise AJ_DEVERR_OFFSETS (that group is left
 * unwritten). */
int aj_grpo_advantages(int32_t n_groups, const int32_t *group_off, const float *reward,
                       float eps, float *ep_adv, uint8_t *ep_keep, int32_t *err, void *stream);

/* A compacted copy of timelines: capacities are the input's sizes
 * (traj_tl_off n_traj+1, tl_tok_off n_tl+1, per-token arrays n_tok). */
typedef struct {
  int32_t *traj_tl_off;
  int64_t *tl_tok_off;
  int32_t *tok;
  uint8_t *flags;
  float *old_logprob;
  float *adv;
  int64_t *counts;              /* [3] episodes, timelines, tokens kept */
} aj_timelines_out;

size_t aj_select_workspace_bytes(int32_t n_traj, int32_t n_tl);
/* Keeps the episodes e with keep[e] != 0, in order, with their timelines and
 * tokens; every kept llm token's advantage becomes ep_adv[e] (the episode's
 * outcome advantage on all of its responses), 0 on the other tokens.
 * in->adv is not read.  Offsets must tile as for aj_merge_timelines
 * (checked on the device: AJ_DEVERR_OFFSETS and counts 0 otherwise). */
int aj_select_episodes(const aj_timelines *in, const uint8_t *keep, const float *ep_adv,
                       aj_timelines_out *out, int32_t *err, void *ws, size_t ws_bytes,
                       void *stream);

/* AdamW with decoupled weight decay (Loshchilov and Hutter) on n float32
 * master parameters; step (4) of Section 4.2 runs optimizer steps after the
 * loss (the optimizer is not named).  With t = step >= 1:
 *   g = grad * grad_scale
 *   m = beta1 m + (1 - beta1) g;   v = beta2 v + (1 - beta2) g^2
 *   param -= lr * weight_decay * param + lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * param_copy (optional, n elements of copy_dtype, an aj_dtype) receives the
 * updated parameters in the storage dtype the forward reads.  Elementwise;
 * any n >= 0; pointers need no alignment. */
int aj_adamw_step(int64_t n, float *param, const float *grad, float *m, float *v, float lr,
                  float beta1, float beta2, float eps, float weight_decay, int32_t step,
                  float grad_scale, void *param_copy, int copy_dtype, void *stream);

/* ------------------------------------------------------------------ timing
 * Benchmark instrumentation.  While enabled, every launch of the kernel
 * classes below is bracketed by two hipEvents recorded on the launch's own
 * stream.  The record is process-wide (the one piece of state the library
 * keeps besides the error text) and meant for a single-threaded driver.
 *   AJ_KC_MERGE      one aj_merge_timelines / aj_merge_timelines_text / aj_flatten_timelines call
 *   AJ_KC_GEMM_*     the MFMA GEMM, by operand layout (NT: both K-major;
 *                    NN: B N-major; TN: A M-major and B N-major), 8-wave
 *                    kernel (reductions shorter than 4096 per split)
 *   AJ_KC_GEMM4_*    the same layouts, 4-wave kernel (longer reductions)
 *   AJ_KC_ATTN_FWD / AJ_KC_ATTN_BWD   the attention kernels of one call
 *   AJ_KC_LM_FWD     the fused logits + log-sum-exp kernel of the LM head
 *   AJ_KC_LM_DZ      the fused logits-recompute + d logits kernel (one per chunk)
 *   AJ_KC_ADAMW      one aj_adamw_step call
 *   AJ_KC_SELECT     one aj_grpo_advantages or aj_select_episodes call
 *   AJ_KC_STAGE_BLOCK  one whole aj_varlen_block_* / aj_stack_* call (the
 *                    decoder-block stage, forward or backward)
 *   AJ_KC_STAGE_LOSS one whole aj_logprob_pg_loss_fwd / _bwd call (the LM
 *                    head and loss stage)
 * The two stage classes span every launch of their call, so they overlap
 * the kernel classes above.  `flops` accumulates algorithmic flops where the
 * library knows them (2*M*N*K per GEMM and LM_FWD launch; 0 for LM_DZ, which
 * recomputes a forward product, and for the other classes). */
enum { AJ_KC_MERGE = 0, AJ_KC_GEMM_NT = 1, AJ_KC_GEMM_NN = 2, AJ_KC_GEMM_TN = 3,
       AJ_KC_ATTN_FWD = 4, AJ_KC_ATTN_BWD = 5, AJ_KC_LM_FWD = 6, AJ_KC_LM_DZ = 7,
       AJ_KC_GEMM4_NT = 8, AJ_KC_GEMM4_NN = 9, AJ_KC_GEMM4_TN = 10, AJ_KC_ADAMW = 11,
       AJ_KC_SELECT = 12, AJ_KC_STAGE_BLOCK = 13, AJ_KC_STAGE_LOSS = 14, AJ_KC_COUNT = 15 };
/* on != 0 starts recording (clearing any earlier record); 0 stops. */
int aj_timing_enable(int on);
/* Waits for every recorded event; fills ms, launches and flops, each [AJ_KC_COUNT]. */
int aj_timing_read(double *ms, int64_t *launches, double *flops);

/* dst[c][r] = src[r][c] for a row-major bfloat16 matrix src [rows, cols]
 * (device pointers, no overlap): the transposed weight copies above.
 * Errors: AJ_ERR_NULL, AJ_ERR_SHAPE (rows or cols < 1). */
int aj_transpose_bf16(const void *src, int32_t rows, int32_t cols, void *dst, void *stream);

/* Measured ceilings of the current device, for reading the rooflines against
 * what the chip sustains as well as its published peaks (bench reporting;
 * nothing on the path calls them).  Both wait for their kernels.
 *   aj_ceiling_mfma_bf16: v_mfma_f32_32x32x16_bf16 from registers only, 8
 *     independent accumulators per wave, one wave per SIMD, with random
 *     bfloat16 operands (random_operands != 0: every product's inputs
 *     toggle, as with trained or random weights) or constant ones; *tflops
 *     is the best of 3 runs.  out: device scratch of at least
 *     2 * CUs * 256 floats (AJ_ERR_WORKSPACE otherwise).
 *   aj_ceiling_copy: a streaming copy of bytes / 2 from the first half of
 *     buf (device, 16-byte aligned, 32 bytes to 1 TiB) to the second, one
 *     16-byte item per thread, then a read-only stream of the first half;
 *     *gbps counts read + write bytes of the copy, *read_gbps the bytes read;
 *     best of 3 runs each after a first one.
 * Errors: AJ_ERR_NULL, AJ_ERR_SHAPE, AJ_ERR_HIP. */
int aj_ceiling_mfma_bf16(int random_operands, void *out, size_t out_bytes, void *stream,
                         double *tflops);
int aj_ceiling_copy(void *buf, size_t bytes, void *stream, double *gbps, double *read_gbps);

#ifdef __cplusplus
}
#endif
#endif /* AJ_H */
