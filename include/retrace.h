/*
 * retrace.h -- C ABI of one ReTrace speculative-decoding round on an MI355X (gfx950).
 *
 * The library runs the round of Algorithm 1 of the ReTrace paper for a batch of
 * independent sequences, every step on the GPU:
 *   1. rejected-trajectory conditioning: alignment (Eq.5, Eq.6), target-aware
 *      correction (Eq.7, Eq.8) and gated residual fusion (Eq.9) of the previous
 *      round's rejected suffix into the next draft block's inputs;
 *   2. the block drafter (DFlash-style: one pass over the anchor and B mask rows,
 *      reading a context KV cache fed by captured target states);
 *   3. the target's block verification (Qwen3-style decoder over a paged KV cache);
 *   4. greedy prefix acceptance, commit of the accepted drafts plus the target's
 *      correction token, KV rollback, and the one-round carry / reset rule.
 * Under greedy verification the committed stream equals the target's own greedy
 * decoding (Section 4, "Optimization and Inference": verification is unchanged).
 *
 * Conventions for every call:
 *  - Return value: RT_OK (0) or a negative RT_ERR_* code; rt_last_error() then
 *    returns a thread-local message.  No C++ exception crosses this boundary.
 *  - Host pointers are owned by the caller and only accessed during the call.
 *  - The device workspace and the HIP stream are owned by the caller and must stay
 *    alive until rt_destroy.  The library owns the layout inside the workspace.
 *  - Calls on one handle must not overlap; separate handles are independent.
 */
#ifndef RETRACE_H
#define RETRACE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  RT_OK = 0,
  RT_ERR_INVALID = -1,    /* malformed argument or configuration */
  RT_ERR_STATE = -2,      /* call out of order (e.g. rt_spec_round before rt_prefill) */
  RT_ERR_CAPACITY = -3,   /* batch, sequence length or budget beyond the configured maxima */
  RT_ERR_WORKSPACE = -4,  /* workspace smaller than rt_workspace_bytes() or misaligned */
  RT_ERR_HIP = -5,        /* a HIP runtime call failed */
  RT_ERR_TOKEN = -6       /* a token id outside [0, vocab) */
};

enum { RT_F32 = 0, RT_BF16 = 1 };                   /* weight / activation storage type */
/* Drafter input conditioning on the previous round's rejected suffix (Section 4.2; the
 * component ablation of Table 3 and its appendix settings):
 *   RT_COND_OFF        plain block drafting: anchor and mask embeddings only;
 *   RT_COND_RETRACE    corrected signal r = m + beta W_c [m; u] (Eq.7-8) fused through the
 *                      gated residual of Eq.9 (the method itself);
 *   RT_COND_RAW_GATED  the same gated residual on the uncorrected signal r = m;
 *   RT_COND_OVERWRITE  the conditioned mask rows are replaced by m_j itself;
 *   RT_COND_LOWRANK    the deployment form of the conditioning path (appendix on
 *                      concurrent serving: rank-64 rejected-suffix latents, input-side
 *                      latent residual fusion, rank-32 target-aware correction), read as
 *                      rho = A m + beta C_up C_down [m; u] and
 *                      e~ = e + (V rho) * sigmoid(W_g[:, :d] e + G rho); its five factors
 *                      follow the other weights (see rt_init_models).
 * Every mode tracks r and cond_len the same way; OFF ignores them. */
enum { RT_COND_OFF = 0, RT_COND_RETRACE = 1, RT_COND_RAW_GATED = 2, RT_COND_OVERWRITE = 3, RT_COND_LOWRANK = 4 };

#define RT_MAX_COND_LAYERS 8

typedef struct rt_config {
  /* Target (Qwen3-style): vocab, hidden d, layers, query / KV heads, head dim, FFN. */
  int32_t vocab, hidden, n_layers, n_q_heads, n_kv_heads, head_dim, ffn;
  float rope_theta;        /* RoPE base (1e6 for Qwen3) */
  float rms_eps;           /* RMSNorm epsilon (1e-6) */
  /* Drafter: layers of the target's width; its context pathway reads the target's
   * residual stream after each listed layer (0-based). */
  int32_t draft_layers, n_cond_layers, cond_layer_ids[RT_MAX_COND_LAYERS];
  int32_t block_size;      /* rows per draft block, anchor included: B = block_size - 1 proposals */
  int32_t mask_token_id;   /* token whose embedding fills the B proposal rows */
  float beta;              /* correction strength of Eq.8 (1.0 at inference) */
  int32_t cond_mode;       /* one of RT_COND_OFF / _RETRACE / _RAW_GATED / _OVERWRITE / _LOWRANK */
  int32_t dtype;           /* RT_BF16 (fp16 retained states) or RT_F32 (fp32 everywhere) */
  int32_t max_batch;       /* sequences per batch */
  int32_t max_seq_len;     /* per sequence: prompt + generation budget + block_size */
  int32_t page_size;       /* KV page size in tokens; must be 16 */
  /* Decoding (Section 5 settings: temperature 0 = greedy; temperature 1 with top-k 20,
   * top-p 0.95).  temperature > 0 selects speculative sampling: drafts are drawn from
   * the drafter's filtered distribution q, draft i is kept with probability
   * min(1, p_i / q_i) against the target's filtered distribution p, and the first
   * rejection draws its correction from the normalised residual max(0, p - q) (a full
   * block draws a bonus token from the last row), so that committed tokens follow the
   * target's own filtered sampling.  A filtered distribution divides the logits by the
   * temperature, keeps the top_k largest (ties to the lowest id), renormalises, and cuts
   * to the shortest prefix whose cumulative probability reaches top_p.  Draws come from
   * a Philox4x64-10 counter (round, sequence, purpose, position) under key
   * (sample_seed, 0). */
  float temperature;       /* 0 (greedy) or > 0 */
  int32_t top_k;           /* 1..RT_MAX_TOP_K and <= vocab (used when temperature > 0) */
  float top_p;             /* (0, 1] (used when temperature > 0) */
  uint64_t sample_seed;
} rt_config;

#define RT_MAX_TOP_K 64

typedef struct rt_model rt_model;   /* opaque handle */

/* Bytes of device workspace the configuration needs (packed weights, paged target
 * and drafter KV caches, activations, round state).  Returns 0 for an invalid
 * configuration (see rt_last_error). */
size_t rt_workspace_bytes(const rt_config* cfg);

/* Number of weight tensors rt_init_models expects for cfg:
 * 1 + 11*n_layers + 4 + 11*draft_layers + 1 + 3, plus 5 with RT_COND_LOWRANK. */
int32_t rt_weight_count(const rt_config* cfg);

/* Elements of weight tensor `index` (0 .. rt_weight_count() - 1) in the order listed at
 * rt_init_models, for the configuration; 0 for an invalid configuration or index. */
int64_t rt_weight_elements(const rt_config* cfg, int32_t index);

/* Builds a model in `d_workspace` (device memory, >= rt_workspace_bytes, 256-byte
 * aligned) on `hip_stream` (a hipStream_t; NULL = default stream).
 *
 * `weights` holds rt_weight_count() pointers, each a row-major [out][in] tensor of the
 * storage type (bf16 bit patterns or float) in device memory or in host memory
 * (pageable or pinned; such tensors are uploaded through temporary device copies,
 * released before the call returns), in this order:
 *   embed [V][d];
 *   per target layer: input_norm [d], q_proj [Hq*hd][d], k_proj [Hkv*hd][d],
 *     v_proj [Hkv*hd][d], q_norm [hd], k_norm [hd], o_proj [d][Hq*hd],
 *     post_norm [d], gate_proj [F][d], up_proj [F][d], down_proj [d][F];
 *   target final_norm [d]; lm_head [V][d] (shared by the drafter);
 *   drafter fc [d][n_cond*d]; drafter hidden_norm [d];
 *   per drafter layer: the same eleven tensors as a target layer;
 *   drafter final_norm [d];
 *   W_c [d][2d] (Eq.7: first d inputs act on m, last d on u);
 *   W_v [d][d] (Eq.9); W_g [d][2d] (Eq.9: first d inputs act on e, last d on r);
 *   with RT_COND_LOWRANK also A [64][d], C_down [32][2d], C_up [64][32], V [d][64],
 *   G [d][64] (W_c and W_v are then unused; W_g's first d columns still act on e).
 * The weights are copied (re-laid out) into the workspace; the caller may free
 * them once the call returns.  The call synchronises the stream. */
int rt_init_models(const rt_config* cfg, const void* const* weights, int32_t n_weights,
                   void* d_workspace, size_t ws_bytes, void* hip_stream, rt_model** out);

/* Runs the target over each prompt (concatenated host token ids, lengths in
 * prompt_lens[n_seqs]), fills the paged target KV cache and the drafter's context
 * KV cache, and returns each sequence's first generated token (greedy) in
 * first_tokens[n_seqs] (host).  gen_budget counts new tokens per sequence, the
 * first one included; prompt_len + gen_budget + block_size must not exceed
 * max_seq_len.  Resets all round state (nothing is carried into round 1). */
int rt_prefill(rt_model* m, int32_t n_seqs, const int32_t* prompt_lens, const int32_t* prompt_ids,
               int32_t gen_budget, int32_t* first_tokens);

/* One ReTrace round for every prefilled sequence.  Outputs (host):
 *   tokens[n_seqs][block_size]: committed tokens of this round, the first
 *     n_committed[s] entries valid (accepted drafts, then the target's correction
 *     or bonus token), -1 elsewhere;
 *   n_committed[n_seqs]: A+1 clipped to the remaining budget; 0 once finished;
 *   accept_len[n_seqs]: A, the number of accepted draft tokens.
 * The rejected-suffix state (retained final drafter / target states, first
 * rejected position, conditioned-row count) stays in the workspace for the next
 * round.  Blocks until the outputs are on the host. */
int rt_spec_round(rt_model* m, int32_t* tokens, int32_t* n_committed, int32_t* accept_len);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): rt_spec_round without any
 * allocation.  The round's kernels are enqueued on the model's stream directly (no
 * HIP graph is instantiated); their partial results -- GEMM split partials and split-K
 * arrival counters, residual k-slab partials, attention key-split partials -- live in a
 * static device array of the library (128 MiB per GPU, held until the process ends)
 * instead of the workspace; the outputs (same meaning and layout as rt_spec_round's)
 * are copied into the caller's DEVICE buffers d_tokens[n_seqs][block_size],
 * d_n_committed[n_seqs] and d_accept_len[n_seqs] on that stream.  Returns once the
 * work is enqueued: the caller synchronises the stream before reading the outputs.
 * Results equal rt_spec_round's bit for bit.  Every allocation-free round on one GPU
 * shares that GPU's array (the split-K counters are cleared at the start of each call
 * by a kernel), so calls that overlap on one GPU -- two models on concurrent streams --
 * race.  Returns RT_ERR_CAPACITY when the configuration's partial results exceed the
 * array, RT_ERR_STATE before rt_prefill or after rt_ar_steps, RT_ERR_HIP if the array's
 * device address could not be obtained when the model was built. */
int rt_spec_round_static(rt_model* m, int32_t* d_tokens, int32_t* d_n_committed, int32_t* d_accept_len);

/* Target-only greedy decoding on the same kernels (the autoregressive baseline that
 * speculative decoding is measured against; Section 5, speedup over target-only
 * decoding).  Each of the n_steps steps (1..RT_AR_MAX_STEPS) runs the target over
 * one row per prefilled sequence -- its last committed token at the next position --
 * appends that row's K/V to the paged cache and commits the argmax of the target's
 * logits.  Outputs (host):
 *   tokens[n_seqs][n_steps]: the committed tokens, -1 once a sequence's budget is spent;
 *   n_generated[n_seqs]: tokens committed by this call.
 * The drafter's context cache is not extended, so after rt_ar_steps only further
 * rt_ar_steps calls are allowed until the next rt_prefill (rt_spec_round returns
 * RT_ERR_STATE).  With debug flag 1 the last step's fp32 logits are kept
 * (RT_T_AR_LOGITS).  Blocks until the outputs are on the host. */
#define RT_AR_MAX_STEPS 256
int rt_ar_steps(rt_model* m, int32_t n_steps, int32_t* tokens, int32_t* n_generated);

/* Releases the handle (the workspace stays the caller's). */
int rt_destroy(rt_model* m);

/* Message for the last non-zero status returned on this thread. */
const char* rt_last_error(void);

/* ---- measurement --------------------------------------------------------------- */

/* Launch classes reported by rt_profile_round (one per role in the round). */
enum {
  RT_K_GEMM_QKV = 0,       /* fused q|k|v projection (target and drafter layers) */
  RT_K_GEMM_O = 1,         /* attention output projection, residual add fused */
  RT_K_GEMM_GATE_UP = 2,   /* fused gate|up projection, SwiGLU fused */
  RT_K_GEMM_DOWN = 3,      /* down projection, residual add (and state capture) fused */
  RT_K_GEMM_CONTEXT = 4,   /* drafter context pathway: fc and the fused context K|V projection */
  RT_K_GEMM_COND = 5,      /* conditioning projections W_c, W_g, W_v (Eq.7-9), fp32 A operand */
  RT_K_ATTENTION = 6,      /* paged attention over key splits (partials or final output) */
  RT_K_ATTN_MERGE = 7,     /* merge of the key-split partials */
  RT_K_NORM = 8,           /* RMSNorm */
  RT_K_QKV_POST = 9,       /* q/k norm, RoPE and paged K/V writes */
  RT_K_LM_HEAD = 10,       /* vocabulary projection with fused argmax */
  RT_K_MISC = 11,          /* embedding gathers, conditioning gather, argmax reduce, acceptance */
  RT_K_KINDS = 12
};
/* Stages of one round, in order (a HIP event at every boundary). */
enum {
  RT_S_CONDITION = 0, RT_S_DRAFT = 1, RT_S_DRAFT_HEAD = 2, RT_S_VERIFY = 3, RT_S_VERIFY_HEAD = 4,
  RT_S_ACCEPT = 5, RT_S_CONTEXT = 6, RT_PROF_STAGES = 7
};
typedef struct rt_kernel_stat {
  int32_t kind;
  int32_t launches;
  double ms;       /* summed kernel execution time (HIP events recorded by each launch) */
  double bytes;    /* summed algorithmic HBM bytes (weights + activations + KV read once) */
  double flops;    /* summed algorithmic FLOPs */
} rt_kernel_stat;

/* Runs one round without graph replay, with a HIP-event pair on every kernel launch
 * on the model's stream and an event at every stage boundary; fills
 * stats[RT_K_KINDS] and stage_ms[RT_PROF_STAGES] plus the usual round outputs.
 * Each kernel's pair is recorded by the launch itself (hipExtLaunchKernel), so the
 * summed times are the kernels' execution times, without host launch gaps. */
int rt_profile_round(rt_model* m, rt_kernel_stat* stats, double* stage_ms, int32_t* tokens,
                     int32_t* n_committed, int32_t* accept_len);

/* Times one launch class in isolation: the launches of `kind` that one round makes
 * (with the round's current buffers and context lengths) are captured into a HIP
 * graph and replayed `reps` times (1..1000) between two HIP events on the model's
 * stream.  stat->launches = launches per round, stat->ms = their summed time per
 * replay (so ms / launches is the kernel's average duration), stat->bytes / flops =
 * their algorithmic totals.  Allowed for RT_K_GEMM_*, RT_K_ATTENTION, RT_K_ATTN_MERGE
 * and RT_K_LM_HEAD, whose outputs are per-round scratch; KV caches and the carried
 * round state are not touched.  Other kinds return RT_ERR_INVALID. */
int rt_time_kernel(rt_model* m, int32_t kind, int32_t reps, rt_kernel_stat* stat);

/* The plain-read ceiling against which the round's weight-streaming kernels are
 * compared: `reps` (1..1000) back-to-back launches of a kernel that reads `bytes` (a
 * positive multiple of 16, at most buf_bytes) of the device buffer d_buf (256-byte
 * aligned, buf_bytes long) once with non-temporal 16-byte loads, each of `grid`
 * (1..65536) workgroups of 256 threads reading one contiguous share,
 * between two HIP events on hip_stream (a hipStream_t; NULL = default stream).
 * Launch r reads the window starting at ((r + 1) * bytes) mod (buf_bytes - bytes + 1)
 * rounded down to 256 bytes, so that with buf_bytes well above the 256 MB memory-side
 * cache every launch reads data that is not cached, as the round's weight streams do.
 * *us = the average duration in microseconds (one warm-up launch first).  Nothing is
 * written.  Needs no model. */
int rt_stream_read(const void* d_buf, size_t buf_bytes, size_t bytes, int32_t grid, int32_t reps, void* hip_stream,
                   double* us);

/* ---- test hooks -------------------------------------------------------------- */

/* Debug flags: 1 = store fp32 logits of both LM heads; 2 = run rounds without
 * HIP-graph replay; 4 = split the reduction of every GEMM four ways (exercises the
 * split-K path on small models); 8 = layer trace: rounds run without graph replay and
 * keep, for every drafter and target layer, its residual input, q, attention output,
 * post-attention residual, post-attention norm output and SwiGLU product, and both LM
 * heads' input operands (RT_T_TRACE_*), so each step can be checked on its own inputs.
 * Setting flag 8 the first time allocates the trace buffer on the device (released by
 * rt_destroy), about (draft_layers + n_layers + 2) x max_batch x block_size x
 * (10 hidden + 4 Hq*hd + 2 ffn) bytes for bf16.  Returns RT_ERR_HIP if that
 * allocation fails.  16 = apply the q / k-norm and RoPE and write the block's K / V
 * rows with the separate post-processing kernel in rounds and target-only steps too
 * (by default the bf16 attention kernel does it there; both round identically).
 * 64 = batches whose attention does not take the q / k work use the spanning key-split
 * plan whenever it is valid (by default only where it shortens the longest split). */
int rt_set_debug(rt_model* m, int32_t flags);

/* Like rt_spec_round, but the verify pass uses drafts[n_seqs][block_size-1] (host)
 * instead of the drafter's argmax (the drafter still runs and its states are
 * still carried). */
int rt_spec_round_forced(rt_model* m, const int32_t* drafts, int32_t* tokens, int32_t* n_committed,
                         int32_t* accept_len);

enum {
  RT_T_DRAFT_LOGITS = 0,   /* [block][V] f32 (needs debug flag 1) */
  RT_T_VERIFY_LOGITS = 1,  /* [block][V] f32 (needs debug flag 1) */
  RT_T_HD = 2,             /* [block][d] retained drafter final states (fp16 or f32) */
  RT_T_HT = 3,             /* [block][d] retained target final states (fp16 or f32) */
  RT_T_ETILDE = 4,         /* [block][d] f32 conditioned drafter inputs */
  RT_T_DRAFT_TOKENS = 5,   /* [block] int32: anchor, then the B draft tokens */
  RT_T_TARGET_TOKENS = 6,  /* [block] int32: target argmax of verify rows 0..B */
  RT_T_STATE = 7,          /* [9] int32: seq_len, anchor, r, cond_len, budget, round_pos, append, A,
                              rounds (or target-only steps) completed */
  RT_T_G = 8,              /* [block][n_cond*d] captured conditioning-layer states (storage type) */
  RT_T_AR_LOGITS = 9,      /* [V] f32 logits of the last rt_ar_steps step (needs debug flag 1 or sampling) */
  /* sampling (temperature > 0): filtered distributions of the last round, [block][RT_MAX_TOP_K],
   * ids in decreasing probability (-1 past the kept entries) and their probabilities */
  RT_T_DRAFT_DIST_IDS = 10,   /* int32, drafter rows (row 0, the anchor row, is not used) */
  RT_T_DRAFT_DIST_P = 11,     /* f32 */
  RT_T_VERIFY_DIST_IDS = 12,  /* int32, target rows 0..B */
  RT_T_VERIFY_DIST_P = 13,    /* f32 */
  RT_T_TARGET_K = 100,     /* + layer: [pos][Hkv][hd] storage type, positions 0.. */
  RT_T_TARGET_V = 200,     /* + layer */
  RT_T_DRAFT_K = 300,      /* + drafter layer: context keys */
  RT_T_DRAFT_V = 400,      /* + drafter layer */
  /* layer trace of the last round (debug flag 8), [block][d] per sequence: */
  RT_T_TRACE_DRAFT_X = 500,   /* + l, l = 0..draft_layers: f32 residual input of drafter layer l
                                 (l = draft_layers: the residual entering the final norm) */
  RT_T_TRACE_TARGET_X = 600,  /* + l, l = 0..n_layers: the same for the verify pass */
  RT_T_TRACE_DRAFT_HEAD = 700,  /* drafter LM-head input (final-norm output, storage type) */
  RT_T_TRACE_VERIFY_HEAD = 701, /* verify LM-head input (storage type) */
  /* + l (drafter layer l); the same items of target layer l are at + 1000 + l: */
  RT_T_TRACE_DRAFT_Q = 1100,    /* [block][Hq*hd] q after q-norm and RoPE (storage type) */
  RT_T_TRACE_DRAFT_ATTN = 1200, /* [block][Hq*hd] attention output (storage type) */
  RT_T_TRACE_DRAFT_XMID = 1300, /* [block][d] f32 residual after the attention block */
  RT_T_TRACE_DRAFT_H2 = 1400,   /* [block][d] post-attention RMSNorm output (storage type) */
  RT_T_TRACE_DRAFT_MLP = 1500,  /* [block][ffn] SwiGLU product silu(gate) * up (storage type) */
  RT_T_TRACE_TARGET_Q = 2100,
  RT_T_TRACE_TARGET_ATTN = 2200,
  RT_T_TRACE_TARGET_XMID = 2300,
  RT_T_TRACE_TARGET_H2 = 2400,
  RT_T_TRACE_TARGET_MLP = 2500
};
/* Copies `bytes` of tensor `tensor_id` for sequence `seq` to host memory.  Reading a
 * trace tensor before flag 8 was set returns RT_ERR_STATE. */
int rt_debug_read(rt_model* m, int32_t tensor_id, int32_t seq, void* host_dst, size_t bytes);
/* Like rt_debug_read for the KV cache tensors (RT_T_TARGET_K/V, RT_T_DRAFT_K/V + layer),
 * starting at position pos0: `bytes` covers positions pos0.. in the [pos][Hkv][hd]
 * layout.  Other tensors return RT_ERR_INVALID. */
int rt_debug_read_rows(rt_model* m, int32_t tensor_id, int32_t seq, int32_t pos0, void* host_dst, size_t bytes);
/* Overwrites RT_T_HD, RT_T_HT, RT_T_STATE, or KV cache rows from position 0
 * (RT_T_TARGET_K/V, RT_T_DRAFT_K/V + layer, [pos][Hkv][hd] storage type) of sequence
 * `seq` from host memory (state injection for tests: a round can then start from a state
 * computed elsewhere). */
int rt_debug_write(rt_model* m, int32_t tensor_id, int32_t seq, const void* host_src, size_t bytes);

#ifdef __cplusplus
}
#endif
#endif /* RETRACE_H */
