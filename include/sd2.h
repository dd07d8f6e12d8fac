/*
 * sd2.h -- C ABI of the MI355X (gfx950) SD^2 speculative-decoding round.
 *
 * One round of SD^2 ("Steering Pretrained Drafters during Speculative
 * Decoding", Berdoz, Rheinboldt, Wattenhofer) on one GPU:
 *   1. the drafter proposes k tokens autoregressively, every processed token's
 *      input embedding carrying the current steering vector s
 *      (Sec. "Drafting": the steering term is computed once per drafting stage
 *      since it does not depend on the draft position, and it also conditions
 *      the keys/values the drafter caches);
 *   2. the verifier scores the block [last committed token, k drafts] in one
 *      parallel forward (Sec. "Verification");
 *   3. speculative rejection sampling (Leviathan et al. 2023, cited in Sec.
 *      "Verification") accepts a prefix of n drafts and draws one final token,
 *      so the block yields n + 1 tokens (Sec. "Metrics", block efficiency);
 *   4. the steering vector for the next round is W_s applied to the verifier's
 *      final-norm hidden state at the position of the last token returned
 *      (Sec. "Verification"); cache lengths roll back to the accepted prefix.
 *
 * Conventions for every call:
 *  - All pointers named "device" are HIP device pointers owned by the caller;
 *    they must stay valid until sd2_destroy.  The library allocates no device
 *    memory: all state lives in the caller's workspace.
 *  - Calls are asynchronous on the HIP stream given to sd2_create, except
 *    sd2_debug_read, which synchronises that stream.  Argument and capacity
 *    errors are detected on the host and returned before anything is enqueued.
 *    HIP errors are returned as SD2_ERR_HIP by the call that observes them.
 *  - A handle is not thread-safe; use one handle per stream.  No C++ exception
 *    crosses this interface.
 *  - Weight matrices are row-major [out][in] ("W x" layout), untied LM head,
 *    no biases.  bf16 tensors hold bfloat16 bit patterns.
 */
#ifndef SD2_H
#define SD2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sd2_status;
#define SD2_OK 0
#define SD2_ERR_INVALID_ARG (-1)   /* bad shape, pointer, alignment or size */
#define SD2_ERR_CAPACITY (-2)      /* prompt + generation would exceed max_seq_len */
#define SD2_ERR_STATE (-3)         /* e.g. sd2_round before sd2_prefill */
#define SD2_ERR_HIP (-4)           /* a HIP runtime call failed; see sd2_last_error */
#define SD2_ERR_UNSUPPORTED (-5)   /* valid request the library does not handle */

typedef struct sd2_handle* sd2_handle_t;

typedef enum { SD2_F32 = 0, SD2_BF16 = 1 } sd2_dtype;

/* Shape of one SwiGLU decoder (the paper's models all use SwiGLU MLPs, eq. (1)).
 * head_dim = d_model / n_heads must be even and at most 128; n_heads must be a
 * multiple of n_kv_heads (grouped-query attention); d_model, n_heads*head_dim
 * and d_ff must be multiples of 64. */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, d_ff, vocab;
    float rope_theta;  /* rotate-half RoPE base */
    float rms_eps;     /* RMSNorm: x / sqrt(mean(x^2) + eps) * gain */
} sd2_dims;

/* Device pointers of one model, all of the configuration's dtype.
 * layers points to a HOST array of n_layers * 9 device pointers, per layer in
 * the order attn_norm[d], wq[H*hd][d], wk[Hkv*hd][d], wv[Hkv*hd][d],
 * wo[d][H*hd], ffn_norm[d], w_gate[F][d], w_up[F][d], w_down[d][F].  The host
 * array is copied by sd2_create; every device pointer must be 16-byte aligned. */
typedef struct {
    const void* embed;             /* [vocab][d] */
    const void* const* layers;     /* host array of n_layers*9 device pointers */
    const void* final_norm;        /* [d] */
    const void* lm_head;           /* [vocab][d] */
} sd2_weights;

typedef struct {
    sd2_dims verifier, drafter;    /* both models must share the vocabulary */
    sd2_dtype dtype;
    int32_t k;                     /* draft length, 1..32 */
    int32_t max_batch;             /* sequences per round, 1..256 */
    int32_t max_seq_len;           /* capacity per sequence: >= prompt + max_new_tokens + k + 1 */
    int32_t max_new_tokens;        /* generated tokens per sequence; its last round is truncated */
    float temperature;             /* 0 => greedy (argmax drafts, accept iff draft == verifier argmax) */
    uint64_t seed;                 /* Philox4x32-10 key of every random draw */
    int32_t steering;              /* SD2_STEER_INPUT or SD2_STEER_NONE (sd2_create); SD2_STEER_MLP,
                                      SD2_STEER_MLP_OUT or SD2_STEER_MLP_COND (sd2_create_mlp) */
    int32_t cond_rank;             /* SD2_STEER_MLP_COND: hidden width R of the conditional bias MLP,
                                      a multiple of 16 in 16..4096; ignored by the other forms */
} sd2_config;

/* How the drafter is steered by the verifier (sd2_config.steering). */
#define SD2_STEER_INPUT 0  /* s = W_s hF (verifier final-norm hidden state, d_V -> d_D) added to the
                              drafter's input embedding of every token it processes in the round */
#define SD2_STEER_MLP 1    /* the paper's eq. (2): g = LayerNorm(W_hml [h; m; l]) from the verifier's
                              residual stream after decoder blocks L_V-2, floor(L_V/2) and 3 (counted
                              from 1; high, middle, low; training details) and one bias b_l = W_s^(l) g
                              per drafter layer, added to the up projection before the gating product:
                              W_d((W_u a + b_l) * SiLU(W_g a)).  Needs L_V >= 3. */
#define SD2_STEER_MLP_OUT 2 /* the paper's ablation "Inv. bias after MLP" (Sec. Ablation): the same g,
                              and one bias b = W_s g of d_D values added to the output of every
                              drafter MLP (x += W_d(...) + b).  Needs L_V >= 3. */
#define SD2_STEER_MLP_COND 4 /* the paper's ablation "Cond. bias in MLP" (Sec. Ablation; its formula is
                              this library's reading): the same g, and per drafter layer l and token
                              the bias U_l SiLU(V_l [f; g]) added to the up projection as in eq. (2),
                              f the residual stream entering layer l at the token's position (the
                              embedding for l = 0), V_l [R][d_D + d_V], U_l [d_ff_D][R].  The g part
                              V_l^g g is computed once per round.  Runs one kernel per operation
                              (no persistent launches).  Needs L_V >= 3. */
#define SD2_STEER_NONE 3   /* no steering: the pretrained drafter the paper compares against (Table 1,
                              "Pretrained"); no steering projection runs and nothing is added to the
                              drafter.  Gives the same outputs as SD2_STEER_INPUT with W_s = 0, without
                              its cost; the baseline of the steering-overhead measurement. */

/* Weights of SD2_STEER_MLP, device pointers in the configuration's dtype, 16-byte aligned. */
typedef struct {
    const void* w_s;       /* SD2_STEER_MLP: [L_D * d_ff_D][d_V], rows l*d_ff_D .. (l+1)*d_ff_D - 1 give
                              layer l's bias; SD2_STEER_MLP_OUT: [d_D][d_V]; SD2_STEER_MLP_COND: V^g
                              [L_D * R][d_V], rows l*R .. (l+1)*R - 1 the g columns of V_l */
    const void* w_hml;     /* [d_V][3 d_V]: g = W_hml [h; m; l] (columns: h, then m, then l) */
    const void* ln_gain;   /* [d_V] LayerNorm gain */
    const void* ln_bias;   /* [d_V] LayerNorm shift */
    float ln_eps;          /* LayerNorm: (g - mean) / sqrt(var + eps) * gain + shift, population variance */
    const void* w_cf;      /* SD2_STEER_MLP_COND: V^f [L_D * R][d_D], the f columns of V_l (else unused) */
    const void* w_cu;      /* SD2_STEER_MLP_COND: U [L_D * d_ff_D][R], rows l*d_ff_D .. the U_l block */
} sd2_mlp_steering;

/* Bytes of device workspace sd2_create needs for cfg (0 if cfg is invalid). */
size_t sd2_workspace_bytes(const sd2_config* cfg);

/*
 * Create a handle.  verifier/drafter: model weights; w_steer: device [d_drafter][d_verifier]
 * steering projection W_s (s = W_s h, paper Sec. "Verification"/"Drafting"), ignored (may be
 * NULL) when cfg->steering is SD2_STEER_NONE;
 * workspace: device buffer of at least sd2_workspace_bytes(cfg) bytes, 256-byte aligned;
 * hip_stream: the hipStream_t every call enqueues on (NULL = default stream).
 * On success *out receives the handle.  Enqueues small table-initialisation kernels.
 * The current HIP device must be a gfx950 (MI355X) with XNACK off, its default mode: the
 * kernels are built for exactly that target, and any other device gives SD2_ERR_UNSUPPORTED
 * (SD2_ERR_HIP if the device cannot be queried).
 */
sd2_status sd2_create(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                      const void* w_steer, void* workspace, size_t workspace_bytes, void* hip_stream,
                      sd2_handle_t* out);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, serving loops
 * and harnesses that forbid hipMalloc): sd2_create with the workspace taken from a static device
 * array of the library instead of the caller.  Allocates nothing, on host or device: the array
 * (SD2_NOALLOC_WORKSPACE_BYTES per GPU) is part of the library's code object, reserved on every
 * GPU the library runs on until the process ends, and the handle's host state sits in a static
 * slot of that GPU.  cfg->steering must be SD2_STEER_INPUT or SD2_STEER_NONE; the other arguments
 * are as sd2_create's, and the handle is used and destroyed the same way.
 * Limits and errors: SD2_ERR_CAPACITY when sd2_workspace_bytes(cfg) exceeds
 * SD2_NOALLOC_WORKSPACE_BYTES (checked before any device call); one such handle per GPU at a
 * time: SD2_ERR_STATE while another one on the current device is alive.  The array keeps the
 * previous handle's contents; creation clears what this handle uses with a kernel (no
 * hipMemsetAsync) on hip_stream, and sd2_destroy of such a handle waits for its stream, so the
 * next handle never clears memory still in use.  Work of a handle from this entry point and any
 * other user of the same array must not overlap on one GPU: they would race on it.
 */
#define SD2_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
sd2_status sd2_create_noalloc(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                              const void* w_steer, void* hip_stream, sd2_handle_t* out);

/*
 * Create a handle whose drafter is steered by the paper's MLP biases (eq. (2); Sec.
 * "Verification" and "Drafting"): cfg->steering must be SD2_STEER_MLP (or SD2_STEER_MLP_OUT, the
 * ablation with one bias after every MLP, or SD2_STEER_MLP_COND, the conditional bias).  Everything else is as
 * sd2_create.  The bias is recomputed at the end of every round from the verifier row whose
 * logits produced the final token, and used for every drafter token of the next round;
 * the drafter processes the prompt without steering, and the first round's bias comes from
 * the verifier at position len-2 (zero when len == 1).
 */
sd2_status sd2_create_mlp(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                          const sd2_mlp_steering* steering, void* workspace, size_t workspace_bytes,
                          void* hip_stream, sd2_handle_t* out);

/*
 * Prefill `batch` sequences (1..max_batch) with their prompts.
 * tokens: device int32 [batch][max_prompt], row b holding lens[b] prompt ids in [0, vocab);
 * lens: device int32 [batch], each in [1, max_prompt]; max_prompt: host bound on lens.
 * Both models process positions 0..len-2 (the drafter with zero steering); the first
 * round's steering vector is W_s applied to the verifier's final-norm hidden state at
 * position len-2 (zero when len == 1).  Returns SD2_ERR_CAPACITY when
 * max_prompt + max_new_tokens + k + 1 > max_seq_len.  Resets all per-sequence state.
 */
sd2_status sd2_prefill(sd2_handle_t h, int32_t batch, const int32_t* tokens, const int32_t* lens,
                       int32_t max_prompt);

/*
 * One speculative round for every prefilled sequence.
 * out_tokens: device int32 [batch][k+1]: row b gets the accepted drafts followed by the
 *             final token (only the first out_counts[b] entries are meaningful);
 * out_counts: device int32 [batch]: tokens emitted this round (n+1, truncated at the
 *             max_new_tokens budget), 0 once the sequence has finished.
 * Returns SD2_ERR_STATE before sd2_prefill.
 */
sd2_status sd2_round(sd2_handle_t h, int32_t* out_tokens, int32_t* out_counts);

/*
 * Test hook: like sd2_round, but the trajectory follows caller-supplied decisions.
 * forced: device int32 [batch][k+2] = k drafts, accepted count n, final token y per
 * sequence.  The library still computes its own decisions from its own logits and
 * records them (sd2_debug_read SD2_DBG_OWN_*); drafting, verification, commit and
 * steering then proceed with the forced values.
 */
sd2_status sd2_round_forced(sd2_handle_t h, const int32_t* forced, int32_t* out_tokens, int32_t* out_counts);

/*
 * Training-objective forward (paper Sec. "Training"; input-form steering, SD2_STEER_INPUT only):
 * for one token sequence x_0..x_{n-1} (tokens: device int32 [n], ids in [0, vocab)) and the
 * offset of every target (deltas: device int32 [n], deltas[tau] in 1..k, entry 0 unused; the
 * paper draws them uniformly), writes out_kl (device float [n]):
 *   out_kl[tau] = KL(p_V || p_D) = sum_v p_V(v) (log p_V(v) - log p_D(v)),  tau = 1..n-1,
 * p_V the verifier's softmax at position tau-1 and p_D the drafter's, whose input embedding at
 * every position p carries the steering of the target it predicts, s_{p+1} = W_s hF_V(p -
 * deltas[p+1]) (zero when that position is negative or the offset lies outside 1..k; hF_V = the
 * verifier's final-norm hidden state), and out_kl[0] = 0; out_loss (device float [1]) receives the mean over tau = 1..n-1.
 * Both models run rows_per_chunk positions at a time (1..512) in sequence slot 0 of the
 * handle's caches, so the handle's generation state is lost (sd2_prefill before the next round).
 * scratch: device buffer of at least sd2_train_loss_scratch_bytes(cfg, n, rows_per_chunk)
 * bytes, 256-byte aligned, caller-owned.  Errors: SD2_ERR_UNSUPPORTED for the MLP and unsteered
 * forms, SD2_ERR_CAPACITY when n > max_seq_len, SD2_ERR_INVALID_ARG otherwise.
 */
size_t sd2_train_loss_scratch_bytes(const sd2_config* cfg, int32_t max_len, int32_t rows_per_chunk);
sd2_status sd2_train_loss(sd2_handle_t h, const int32_t* tokens, const int32_t* deltas, int32_t n,
                          int32_t rows_per_chunk, float* out_kl, float* out_loss, void* scratch,
                          size_t scratch_bytes);

/* Destroy a handle (NULL is a no-op).  Does not free caller memory. */
sd2_status sd2_destroy(sd2_handle_t h);

/* Static text for a status code. */
const char* sd2_status_string(sd2_status s);

/* Text of the last HIP error observed by handle h (empty if none). */
const char* sd2_last_error(sd2_handle_t h);

/* What sd2_debug_read copies (all host-side, after synchronising the stream). */
#define SD2_DBG_LOGITS_V 1    /* float [batch][k+1][vocab]: last round's verifier logits */
#define SD2_DBG_LOGITS_D 2    /* float [batch][k][vocab]: last round's drafter logits (row j drew draft j) */
#define SD2_DBG_STEER 3       /* float [batch][d_drafter]: current steering vector s (SD2_STEER_INPUT) */
#define SD2_DBG_OWN_DRAFTS 4  /* int32 [batch][k]: drafts the library drew itself last round */
#define SD2_DBG_OWN_N 5       /* int32 [batch]: accepted count the library computed itself */
#define SD2_DBG_OWN_Y 6       /* int32 [batch]: final token the library drew itself */
#define SD2_DBG_STATE 7       /* int32 [batch][5]: t, len_verifier, len_drafter, produced, done */
#define SD2_DBG_HIST 8        /* int32 [batch][max_seq_len]: committed tokens */
#define SD2_DBG_HIDDEN_V 9    /* float [batch][k+1][d_verifier]: last verify pass's final-norm hidden states */
#define SD2_DBG_PATH 10       /* int32 [2]: round execution path (0: one kernel per operation, 1: one persistent
                                 launch per drafter step and per verify pass), and 1 if one of those launches
                                 ever timed out at a grid barrier (its results are then invalid) */
#define SD2_DBG_TRACE 11      /* int64 [33][1024]: persistent path, last profiled round, device clock
                                 (100 MHz): entry 0 = start of launch j (0: verify pass, 1..k: drafter
                                 steps), entry p+1 = end of its phase p; SD2_ERR_STATE when that path
                                 is unavailable */

#define SD2_DBG_UBIAS 12      /* float [batch][L_D][d_ff_D]: current up-projection biases (SD2_STEER_MLP),
                                 float [batch][d_D]: the bias after every MLP (SD2_STEER_MLP_OUT);
                                 SD2_ERR_STATE for SD2_STEER_INPUT */
#define SD2_DBG_NONFINITE 13  /* int32 [1]: 1 if a verifier or drafter logit of a round since the last read of
                                 this selector was a NaN or an infinity (every logit the round's decisions use
                                 is checked as the sampler reads it), else 0; the read clears it */

/* Copy a debug buffer of the last round into host memory dst (bytes must match). */
sd2_status sd2_debug_read(sd2_handle_t h, int32_t what, void* dst_host, size_t bytes);

/* Kernel classes for sd2_profile_read. */
#define SD2_PROF_GEMV 1      /* weight-streaming projections and LM heads */
#define SD2_PROF_ATTN 2      /* attention over the KV cache */
#define SD2_PROF_SAMPLER 3   /* draft picks, accept test, final draw, commit */
#define SD2_PROF_OTHER 4     /* embedding/planning, RoPE and cache append */
#define SD2_PROF_PROGRAM 5   /* persistent launches (one per drafter step, one per verify pass) */

/*
 * Measurement hook.  enable != 0: following rounds are launched one kernel at a time (not from
 * the recorded graph) with a HIP event pair recorded on the handle's stream around every
 * launch; enable == 0 returns to graph replay.  Rounds stay functionally identical.
 */
sd2_status sd2_profile(sd2_handle_t h, int32_t enable);

/*
 * For the last profiled round (synchronises the stream): number of launches of class cls,
 * the sum of their event-to-event durations in milliseconds, and the sum of their algorithmic
 * bytes (SD2_PROF_GEMV: weights + input rows + output rows; SD2_PROF_PROGRAM: the weights the
 * launch streams, KV-cache reads not included; 0 for other classes).
 */
sd2_status sd2_profile_read(sd2_handle_t h, int32_t cls, int32_t* launches, double* total_ms, double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* SD2_H */
