// Private host/device interface of the SD^2 engine: workspace layout and kernel launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sd2.h"
#include "mk.h"

namespace sd2 {

constexpr int kMaxK = 32;
constexpr int kVocabChunks = 64;     // vocabulary slices per row in the sampler's partial reductions
constexpr int kPrefillRows = 512;    // rows per prefill chunk (all sequences together)

struct ModelDev {
    sd2_dims dm;
    int hd, qkv_dim;
    const void* embed;
    const void* layer[9 * 128];      // per layer: attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down
    const void* final_norm;
    const void* lm_head;
    // workspace-resident
    float* kc;                        // K cache [layer][batch][kv_head][cap][hd]
    float* vc;                        // V cache, same layout
    float* rope_cos;                  // [cap][hd/2]
    float* rope_sin;
    float* x;                         // residual stream [maxm][d]
    float* ss;                        // [maxm][d/16] sums of squares of 16-column slices of x
};

enum WIdx { kAttnNorm = 0, kWq, kWk, kWv, kWo, kFfnNorm, kWg, kWu, kWd };

// Partial result of a vocabulary slice for one row.
struct VPart {
    float m;     // max of scores
    float s;     // sum of exp(score - m)   (or second field for argmax partials)
    float best;  // best perturbed score
    int idx;     // its token
    float best2; // fallback score (final draw: plain p-Gumbel)
    int idx2;
    int flag;    // final draw: residual had positive mass in this slice
    int pad;
};

struct Workspace {
    // per-sequence state, int32 [max_batch]
    int32_t *t, *len_v, *len_d, *produced, *done;
    int32_t* hist;          // [max_batch][cap]
    float* steer;           // [max_batch][d_D]
    float* hcap;            // [max_batch][d_V] verifier residual captured at prefill
    float* hcap_ss;         // [max_batch][d_V/16] its slice sums of squares
    // row plans
    int32_t* row_pos;       // [maxm]
    int32_t* row_seq;       // [maxm]
    int32_t* lm_map_d;      // [k][2*max_batch] drafter LM-head output rows per step
    int32_t* steer_map;     // [max_batch]
    int32_t* ident_map;     // [2 max_batch] 0..2 max_batch-1
    // activations
    float* qkv;             // [maxm][max qkv_dim]
    float* attn;            // [maxm][max H*hd]
    float* ffh;             // [maxm][max F]
    float* logits_v;        // [max_batch][k+1][V]
    float* logits_d;        // [max_batch][k][V]
    float* hidden_dbg;      // [max_batch*(k+1)][d_V]
    VPart* part;            // [max_batch*(2k+1)][kVocabChunks]
    float* lse_v;           // [max_batch][k+1]
    float* lse_d;           // [max_batch][k]
    int32_t* argmax_v;      // [max_batch][k+1] (greedy)
    // decisions
    int32_t* drafts;        // [max_batch][k] effective drafts
    int32_t* own_drafts;    // [max_batch][k]
    int32_t* n_eff;         // [max_batch]
    int32_t* own_n;
    int32_t* own_y;
    int32_t* forced;        // [max_batch][k+2]
    int32_t* forced_on;     // [1]
    // split-K partial tiles of the projection kernel; attention partials per position span
    float* ws_part;
    int32_t* ws_cnt;
    size_t ws_part_n, ws_cnt_n;  // their capacities (floats, counters)
    float* attn_part;
    int32_t* attn_cnt;
    int32_t* nonfinite;     // set to 1 by the sampler when a logit row it reads holds a NaN or an infinity
    size_t attn_cnt_n;      // its capacity (counters)
    // MLP steering (null unless cfg.steering == SD2_STEER_MLP)
    float* taps;            // [3][maxm][d_V] verifier residual after the tap blocks (per-operation path)
    float* tapsel;          // [max_batch][3 d_V] [h; m; l] of each sequence's steering row
    float* gsteer;          // [max_batch][d_V] g = W_hml [h; m; l], then its LayerNorm
    float* ubias;           // [max_batch][nbias] biases of the current round (L_D x F_D, or d_D; the conditional
                            // bias: the g parts V_l^g g, L_D x R)
    float* cond_h;          // conditional bias: [2 max_batch][R] hidden layer of the drafter rows
    float* cond_b;          // conditional bias: [2 max_batch][F_D] one layer's bias of the drafter rows
};

// Per-launch timing entries (HIP events recorded on the engine's stream).
enum ProfClass { kProfGemv = 1, kProfAttn = 2, kProfSampler = 3, kProfOther = 4, kProfProgram = 5 };
constexpr int kProfMax = 4096;
struct ProfEntry {
    int cls;
    double bytes;
    hipEvent_t a, b;
};

struct Engine {
    sd2_config cfg;
    ModelDev mv, md;
    const void* w_steer;    // SD2_STEER_INPUT: [d_D][d_V]; SD2_STEER_MLP: [L_D*F_D][d_V]; null: SD2_STEER_NONE
    bool mlp;               // cfg.steering is SD2_STEER_MLP or SD2_STEER_MLP_OUT (taps, W_hml, LayerNorm)
    bool bias_after;        // SD2_STEER_MLP_OUT: the bias joins every drafter MLP's output
    bool cond;              // SD2_STEER_MLP_COND: per-row biases U_l SiLU(V_l^f f + V_l^g g) (one kernel per op)
    const void *w_cf, *w_cu;  // SD2_STEER_MLP_COND: V^f [L_D R][d_D], U [L_D F_D][R]
    int nbias;              // bias values per sequence: L_D*F_D or d_D
    const void *w_hml, *ln_gain, *ln_bias;
    float ln_eps;
    int tap_layer[3];       // 0-based verifier layers after which h, m, l are taken
    Workspace ws;
    int cap, maxm, batch;
    bool prefilled;
    hipStream_t stream;
    bool bf16;
    char err[256];
    bool use_graph;
    hipGraphExec_t graph_exec;
    hipGraph_t graph;
    int graph_batch;
    int32_t* graph_out_tokens;
    int32_t* graph_out_counts;
    bool bad_launch;  // a projection shape had no kernel instance (reported as SD2_ERR_UNSUPPORTED)
    hipError_t launch_err;  // failure of a launch call that returns an error (round-program path)
    bool prof_on;
    int prof_n;
    ProfEntry* prof;
    MkState mk;  // persistent round-program path (used when active)
    bool static_slot;   // created by sd2_create_noalloc: workspace and this object are static
    int static_device;  // its device
};

// Size of the static device workspace of sd2_create_noalloc (per GPU).
constexpr size_t kStaticWorkspaceBytes = SD2_NOALLOC_WORKSPACE_BYTES;

// Bracket one launch with timing events when profiling is enabled (no-op otherwise).
void prof_begin(Engine* e, int cls, double bytes);
void prof_end(Engine* e);
// For launches through hipExtLaunchKernelGGL: the next free entry (nullptr when not profiling);
// its events are handed to the dispatch itself, so their span is the kernel's own execution.
ProfEntry* prof_slot(Engine* e, int cls, double bytes);
void prof_commit(Engine* e);

size_t carve(const sd2_config& c, char* base, Workspace* ws, ModelDev* mv, ModelDev* md, int* maxm,
             MkState* mk = nullptr);

// ---- launchers (kernels.hip) ----
void launch_rope_table(hipStream_t s, ModelDev& m, int cap);
void launch_init_maps(hipStream_t s, Engine& e);
enum PlanKind { kPlanDraft1 = 0, kPlanDraftJ = 1, kPlanVerify = 2, kPlanPrefill = 3 };
void launch_plan_embed(hipStream_t s, Engine& e, ModelDev& m, int kind, int j, int rows, const int32_t* prompt_tok,
                       const int32_t* prompt_len, int max_prompt, int chunk, const float* row_add = nullptr);
// ub_map (null: the row's sequence) maps rows to bias rows (the conditional bias: one per row).
// ubias (drafter rounds with MLP steering): this layer's biases, row stride ub_ld, indexed by
// the row's sequence, added to the up projection, or to the MLP output when bias_after; null
// for none.
void launch_layer(hipStream_t s, Engine& e, ModelDev& m, int layer, int rows, int rps, const float* ubias = nullptr,
                  int ub_ld = 0, bool bias_after = false, const int32_t* ub_map = nullptr);
// Conditional bias of drafter layer `layer` for every row: cond_b = U_l SiLU(V_l^f x + c_l[seq]).
void launch_cond_bias(hipStream_t s, Engine& e, int layer, int rows);
// Final-norm LM head of `rows` residual rows into Y[out_map[r]] (bf16 path via the projection kernel).
void launch_lm_head(Engine& e, ModelDev& m, int rows, float* Y, const int32_t* out_map);
void launch_steer(Engine& e, const float* X, const float* ss, const int32_t* in_map, int rows);
// MLP steering: copy the verifier residual rows after `layer` to the tap slots taken there.
void launch_tap_copy(hipStream_t s, Engine& e, int layer, int rows);
// Prefill: keep the tap rows at position len-2 of every sequence (slots taken after `layer`).
void launch_prefill_tap(hipStream_t s, Engine& e, int layer, int rows, const int32_t* prompt_len, int max_prompt);
// Gather [h; m; l] of row in_map[b] from src[3] ([rows][d_V] each) into tapsel, then
// gsteer = LayerNorm(W_hml tapsel) and ubias = W_s gsteer, for `rows` sequences.
void launch_mlp_steer(Engine& e, const float* const* src, const int32_t* in_map, int rows);
enum Epi { kEpiStore = 0, kEpiAdd = 1, kEpiSwiglu = 2, kEpiQkv = 3 };

// One bf16 weight-streaming projection (see wsgemv.hip).
struct WsCall {
    const float* X;
    const int32_t* in_map;
    int M, K;
    const void* gamma;  // RMSNorm gain (bf16) or null
    float eps;
    const float* ss;    // [rows][nss] slice sums of squares of the X rows (norm input)
    int nss;
    const void* W[3];
    int seg_rows[3];
    int nseg, mode;
    float* Y;
    int ldy;
    const int32_t* out_map;
    float* ss_out;
    float* part;
    int32_t* cnt;
    int H, Hkv, hd;
    const int32_t *row_pos, *row_seq;
    const float *rcos, *rsin;
    float *qout, *kc, *vc;
    int cap, max_batch, layer;
    const float* ubias;  // per-sequence bias rows (stride ub_ld, row_seq): SwiGLU adds them to up, Add
                         // to the output; or null
    int ub_ld;
};
struct WsPlan {
    int KR, S, tiles, NW, steps, Gt;
    size_t lds;
};
WsPlan ws_plan(int M, int N, int K, int mode);
void launch_wsgemv(Engine* e, hipStream_t s, const WsCall& c);
hipError_t wsgemv_setup();
int pg_split(int M, int N, int K, int subs);  // K ranges of the many-row GEMM for a shape  // kernel attributes of the many-row GEMM (once per process and device)
void launch_attn(Engine& e, hipStream_t s, ModelDev& m, int layer, int rows, int rps, const float* q, int q_stride);
int attn_nsplit(int cap);
size_t attn_groups(int rows, int rps, int H, int Hkv);
void launch_gemv(Engine* e, hipStream_t s, bool bf16, const float* X, const int32_t* in_map, int M, int K,
                 const void* gamma, float eps, const void* const* W, const int* seg_rows, int nseg, int epi, float* Y,
                 int ldy, const int32_t* out_map, const float* ubias = nullptr, int ub_ld = 0,
                 const int32_t* row_seq = nullptr);
void launch_draft_pick(hipStream_t s, Engine& e, int j);
void launch_verify_decide(hipStream_t s, Engine& e, int32_t* out_tokens, int32_t* out_counts);
void launch_prefill_capture(hipStream_t s, Engine& e, int rows, const int32_t* prompt_len, int max_prompt);
void launch_prefill_finish(hipStream_t s, Engine& e, int batch, const int32_t* prompt_tok, const int32_t* prompt_len,
                           int max_prompt);
void launch_rmsnorm_rows(hipStream_t s, const float* X, int rows, int d, const void* gamma, bool bf16, float eps,
                         float* Y);
void launch_set_flag(hipStream_t s, int32_t* flag, int v);

// Training-objective forward (sd2_train_loss): buffers carved from the caller's scratch.
struct LossScratch {
    float* lv;      // [chunk][V] verifier logits of a chunk
    float* ld;      // [chunk][V] drafter logits of a chunk
    float* hf;      // [nchunks * chunk + 1][d_V] verifier final-norm hidden rows (last: zeros)
    float* srow;    // [chunk][d_D] steering of every target of a chunk
    int32_t* src;   // [chunk] source rows of those steering vectors
    int32_t* len;   // [1] the sequence length
};
void launch_train_loss(hipStream_t s, Engine& e, const int32_t* tokens, const int32_t* deltas, int n, int chunk,
                       const LossScratch& w, float* out_kl, float* out_loss);

}  // namespace sd2
