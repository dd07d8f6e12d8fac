/*
 * oracle.c -- plain, slow CPU reference of one SD^2 speculative-decoding round.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or load
 * this file; only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or constant generator with
 * the GPU library.
 *
 * Arithmetic: float64 throughout the model forward (weights are read as stored,
 * bf16 or f32, and widened exactly to double).  Discrete decisions (draft picks,
 * accept tests, final-token draws) are taken in float32 on float32-rounded
 * logits and log-normalisers, because that is the precision the GPU sampler
 * decides in.  Every sum is a plain sequential loop; a row's arithmetic never
 * depends on how many rows are processed together, so a block of k+1 rows gives
 * bit-identical results to k+1 single-row steps.
 *
 * What it follows (paper: "Steering Pretrained Drafters during Speculative
 * Decoding", Berdoz, Rheinboldt, Wattenhofer):
 *   - model forward: SwiGLU decoder layers, eq. (1) of Sec. "Drafting"
 *     (sigma read as SiLU); RMSNorm, rotate-half RoPE, grouped-query attention.
 *   - drafting: k autoregressive drafter steps conditioned on the steering
 *     vector (Sec. "Drafting"); the steering bias is computed once per drafting
 *     stage because it does not depend on the draft position, and the keys and
 *     values a token writes keep the steering that was active when it was
 *     processed.  Injection point: the steering vector s = W_s h* is added to
 *     the drafter's input embedding of every token processed in the round,
 *     before its first layer.
 *   - verification: the verifier scores all k+1 block positions in one pass
 *     (Sec. "Verification"); accept/reject by speculative rejection sampling
 *     (Leviathan et al. 2023; Chen et al. 2023, cited there): accept draft i
 *     with probability min(1, p_i/q_i), then draw the final token from the
 *     normalised residual (p - q)+ after a rejection or from p_{k+1} when all k
 *     drafts were accepted; the block yields accepted + 1 tokens (Sec.
 *     "Metrics", block efficiency).
 *   - steering tap: the verifier's final-norm hidden state at the row whose
 *     logits produced the final token, i.e. the position of the last token
 *     returned (Sec. "Verification"), projected by W_s.
 *   - MLP steering, the paper's own form (eq. (2), Sec. "Verification" and
 *     "Drafting", Fig. 2, training details): the verifier's residual stream
 *     after decoder blocks L-2, floor(L/2) and 3 (counted from 1; high,
 *     middle, low) at that same row is concatenated as [h; m; l], mapped by
 *     W_hml to g, passed through a LayerNorm (population variance, gain and
 *     shift), and W_s g gives one bias per drafter layer (rows l*F..(l+1)*F of
 *     W_s), added to the up projection before the gating product:
 *     W_d((W_u a + b_l) * SiLU(W_g a)).  The bias is computed once per round
 *     and used for every drafter token processed in that round.
 *   - the ablation "Inv. bias after MLP" (Sec. "Ablation", the simplest of the
 *     three steering mechanisms compared there): the same g, and one bias
 *     W_s g of d_model values added to the output of every drafter MLP.
 *   - the ablation "Cond. bias in MLP" (same paragraph: the bias depends on
 *     g and on the previous layer's output): a two-layer MLP per drafter
 *     layer l, b = U_l SiLU(V_l [f; g]), where f is the residual stream that
 *     enters layer l (the output of layer l-1; the embedding for l = 0) at the
 *     token's own position, V_l [R][d_D + d_V] and U_l [d_ff][R]; b is added to
 *     the up projection as in eq. (2).  V_l [f; g] = V_l^f f + V_l^g g: the
 *     g part is computed once per round (like eq. (2)'s bias), the f part per
 *     token and layer.
 *   - training objective (Sec. "Training"; offset ablation in the appendix):
 *     for a token sequence and per target position tau an offset delta_tau
 *     drawn uniformly from [1, k], the loss is the mean over tau of
 *     KL(pi_V(.|x_<tau) || pi_D(.|x_<tau, g from delta_tau positions back)).
 *     Reading: the steering that predicts x_tau with offset delta is the one a
 *     round starting at tau - delta + 1 uses, W_s hF_V(tau - delta - 1) (zero
 *     before the sequence start); in the one-pass forward every drafter input
 *     position p carries the steering of the target it predicts, x_{p+1}.
 *   - greedy regime (T = 0): argmax drafts, accept iff the draft equals the
 *     verifier's argmax, final token = verifier argmax (Sec. "Decoding
 *     Parameters").
 *   - randomness: Philox4x32-10 (Salmon et al., SC'11), counter keyed by
 *     (index, step, round start t, purpose<<24 | sequence); uniforms use the top
 *     23 bits of a word; Gumbel-max draws
 *     argmax_v(l_v/T + G_v) with G = -log(-log u).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ----------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon et al. 2011): 10 rounds of the 4x32 bijection with  */
/* multipliers 0xD2511F53, 0xCD9E8D57 and Weyl key increments 0x9E3779B9,   */
/* 0xBB67AE85.                                                               */
/* ----------------------------------------------------------------------- */
void oracle_philox(const uint32_t in[4], uint32_t k0, uint32_t k1, uint32_t out[4]) {
    uint32_t x0 = in[0], x1 = in[1], x2 = in[2], x3 = in[3];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t prod_a = (uint64_t)0xD2511F53u * (uint64_t)x0;
        uint64_t prod_b = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
        uint32_t y0 = (uint32_t)(prod_b >> 32) ^ x1 ^ k0;
        uint32_t y1 = (uint32_t)prod_b;
        uint32_t y2 = (uint32_t)(prod_a >> 32) ^ x3 ^ k1;
        uint32_t y3 = (uint32_t)prod_a;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

enum { PURPOSE_DRAFT = 1, PURPOSE_ACCEPT = 2, PURPOSE_FINAL = 3 };

/* 32-bit word `word` of the Philox block at counter (c0, c1, c2, purpose<<24 | b). */
static uint32_t rng_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t purpose,
                         uint32_t b, int word) {
    uint32_t ctr[4] = {c0, c1, c2, (purpose << 24) | b};
    uint32_t out[4];
    oracle_philox(ctr, (uint32_t)seed, (uint32_t)(seed >> 32), out);
    return out[word];
}

/* Uniform in (0,1): the top 23 bits plus one half, times 2^-23; every step is exact
 * in float32, so u lies in [2^-24, 1 - 2^-24]. */
float oracle_uniform(uint32_t w) { return ((float)(w >> 9) + 0.5f) * (1.0f / 8388608.0f); }

float oracle_gumbel(uint32_t w) { return -logf(-logf(oracle_uniform(w))); }

/* Gumbel noise for vocabulary entry v of a draw with counter (c1, c2, purpose, b). */
static float gumbel_at(uint64_t seed, uint32_t v, uint32_t c1, uint32_t c2, uint32_t purpose, uint32_t b) {
    return oracle_gumbel(rng_word(seed, v >> 2, c1, c2, purpose, b, (int)(v & 3)));
}

/* ----------------------------------------------------------------------- */
/* Model description and weight access                                      */
/* ----------------------------------------------------------------------- */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, d_ff, vocab;
    double rope_theta, rms_eps;
} odims;

enum { W_ATTN_NORM = 0, W_Q, W_K, W_V, W_O, W_FFN_NORM, W_GATE, W_UP, W_DOWN, W_PER_LAYER };

typedef struct {
    odims dm;
    int bf16;                  /* 1: weights stored as bf16 bit patterns; 0: float32 */
    const void* embed;         /* [vocab][d] */
    const void** layers;       /* n_layers * 9 pointers, order W_ATTN_NORM..W_DOWN */
    const void* final_norm;    /* [d] */
    const void* lm_head;       /* [vocab][d] */
} omodel;

static inline double wval(int bf16, const void* base, size_t i) {
    if (bf16) {
        uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
        float f;
        memcpy(&f, &bits, 4);
        return (double)f;
    }
    return (double)((const float*)base)[i];
}

/* Y[r][n] = sum_k W[n][k] * X[r][k] for r < rows; the sum runs over k in order. */
static void matmul_rows(int bf16, const void* W, int N, int K, const double* X, int rows, double* Y) {
#pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
        for (int r = 0; r < rows; ++r) {
            const double* x = X + (size_t)r * K;
            double acc = 0.0;
            for (int k = 0; k < K; ++k) acc += wval(bf16, W, (size_t)n * K + k) * x[k];
            Y[(size_t)r * N + n] = acc;
        }
    }
}

/* y = x / sqrt(mean(x^2) + eps) * g */
static void rmsnorm(int bf16, const void* g, int d, double eps, const double* x, double* y) {
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += x[i] * x[i];
    double inv = 1.0 / sqrt(ss / d + eps);
    for (int i = 0; i < d; ++i) y[i] = x[i] * inv * wval(bf16, g, i);
}

/* Rotate-half RoPE on one head vector at absolute position pos. */
static void rope(double* v, int hd, int pos, double theta) {
    int half = hd / 2;
    for (int i = 0; i < half; ++i) {
        double ang = (double)pos * pow(theta, -2.0 * i / hd);
        double c = cos(ang), s = sin(ang);
        double a = v[i], b = v[i + half];
        v[i] = a * c - b * s;
        v[i + half] = b * c + a * s;
    }
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* Per-sequence KV cache: K,V[layer][pos][kv_head][hd] in double. */
typedef struct {
    int cap;
    double* k;
    double* v;
} okv;

static size_t kv_index(const odims* dm, int cap, int layer, int pos, int h) {
    int hd = dm->d_model / dm->n_heads;
    return (((size_t)layer * cap + pos) * dm->n_kv_heads + h) * hd;
}

/* Decoder blocks whose outputs are the steering taps, in the order h, m, l:
 * blocks L-2, floor(L/2) and 3 counted from 1, as 0-based layer indices. */
static void tap_layers(int L, int out[3]) {
    out[0] = L - 3;
    out[1] = L / 2 - 1;
    out[2] = 2;
}

/* Conditional bias in the MLP: per layer l, b = U_l SiLU(Vf_l f + c_l) with
 * c_l = Vg_l g precomputed for the round (rows l*R .. (l+1)*R-1 of c). */
typedef struct {
    const void* vf;            /* [L*R][d]: V_l^f, the columns of V_l that multiply f */
    const void* u;             /* [L*d_ff][R]: U_l */
    int rank;                  /* R */
    const double* c;           /* [L*R]: V_l^g g for this sequence and round */
} ocond;

/*
 * Forward of m consecutive tokens at positions pos0..pos0+m-1 of one sequence
 * whose cache holds positions 0..pos0-1.  `add` (d doubles, may be NULL) is
 * added to every input embedding (the steering injection).  `ubias` (NULL for
 * none) holds one bias of d_ff values per layer, added to the up projection
 * before the gating product (eq. (2)); `obias` (d values, NULL for none) is
 * added to the output of every layer's MLP; `cond` (NULL for none) adds the
 * conditional bias U_l SiLU(V_l [f; g]) of every row to its up projection, f
 * being the row's residual stream as it enters the layer.  `taps` (NULL for none) receives, per
 * row, the residual stream after the three tap blocks: taps[m][3][d].  Writes
 * the final-norm hidden state of every row to hF[m][d] and, when
 * logits != NULL, the logits of every row to logits[m][vocab].
 */
static void forward_block(const omodel* M, okv* kv, int pos0, int m, const int32_t* toks,
                          const double* add, const double* ubias, const double* obias, const ocond* cond,
                          double* taps, double* hF, double* logits) {
    const odims* dm = &M->dm;
    int d = dm->d_model, H = dm->n_heads, Hkv = dm->n_kv_heads, F = dm->d_ff;
    int hd = d / H, group = H / Hkv;
    double* x = calloc((size_t)m * d, sizeof(double));
    double* nrm = calloc((size_t)m * d, sizeof(double));
    double* q = calloc((size_t)m * H * hd, sizeof(double));
    double* kk = calloc((size_t)m * Hkv * hd, sizeof(double));
    double* vv = calloc((size_t)m * Hkv * hd, sizeof(double));
    double* att = calloc((size_t)m * H * hd, sizeof(double));
    double* proj = calloc((size_t)m * d, sizeof(double));
    double* gate = calloc((size_t)m * F, sizeof(double));
    double* up = calloc((size_t)m * F, sizeof(double));
    double* cb = cond ? calloc((size_t)m * F, sizeof(double)) : NULL;          /* [m][F] conditional bias */
    double* ch = cond ? calloc((size_t)m * cond->rank, sizeof(double)) : NULL; /* [m][R] its hidden layer */
    int maxlen = pos0 + m;
    for (int r = 0; r < m; ++r)
        for (int i = 0; i < d; ++i)
            x[(size_t)r * d + i] = wval(M->bf16, M->embed, (size_t)toks[r] * d + i) + (add ? add[i] : 0.0);

    for (int l = 0; l < dm->n_layers; ++l) {
        const void** Wl = M->layers + (size_t)l * W_PER_LAYER;
        if (cond) {
            /* b = U_l SiLU(V_l^f f + V_l^g g), f = x as it enters the layer */
            int R = cond->rank;
            const void* vf = (const char*)cond->vf + (size_t)l * R * d * (M->bf16 ? 2 : 4);
            const void* u = (const char*)cond->u + (size_t)l * F * R * (M->bf16 ? 2 : 4);
            matmul_rows(M->bf16, vf, R, d, x, m, ch);
            for (int r = 0; r < m; ++r)
                for (int i = 0; i < R; ++i)
                    ch[(size_t)r * R + i] = silu(ch[(size_t)r * R + i] + cond->c[(size_t)l * R + i]);
            matmul_rows(M->bf16, u, F, R, ch, m, cb);
        }
        /* attention sub-block */
        for (int r = 0; r < m; ++r) rmsnorm(M->bf16, Wl[W_ATTN_NORM], d, dm->rms_eps, x + (size_t)r * d, nrm + (size_t)r * d);
        matmul_rows(M->bf16, Wl[W_Q], H * hd, d, nrm, m, q);
        matmul_rows(M->bf16, Wl[W_K], Hkv * hd, d, nrm, m, kk);
        matmul_rows(M->bf16, Wl[W_V], Hkv * hd, d, nrm, m, vv);
        for (int r = 0; r < m; ++r) {
            int pos = pos0 + r;
            for (int h = 0; h < H; ++h) rope(q + ((size_t)r * H + h) * hd, hd, pos, dm->rope_theta);
            for (int h = 0; h < Hkv; ++h) {
                rope(kk + ((size_t)r * Hkv + h) * hd, hd, pos, dm->rope_theta);
                memcpy(kv->k + kv_index(dm, kv->cap, l, pos, h), kk + ((size_t)r * Hkv + h) * hd, hd * sizeof(double));
                memcpy(kv->v + kv_index(dm, kv->cap, l, pos, h), vv + ((size_t)r * Hkv + h) * hd, hd * sizeof(double));
            }
        }
#pragma omp parallel for collapse(2) schedule(static)
        for (int r = 0; r < m; ++r) {
            for (int h = 0; h < H; ++h) {
                int pos = pos0 + r, g = h / group;
                const double* qv = q + ((size_t)r * H + h) * hd;
                double* sc = malloc((size_t)maxlen * sizeof(double));
                double mx = -INFINITY;
                for (int j = 0; j <= pos; ++j) {
                    const double* kj = kv->k + kv_index(dm, kv->cap, l, j, g);
                    double dot = 0.0;
                    for (int i = 0; i < hd; ++i) dot += qv[i] * kj[i];
                    sc[j] = dot / sqrt((double)hd);
                    if (sc[j] > mx) mx = sc[j];
                }
                double den = 0.0;
                for (int j = 0; j <= pos; ++j) {
                    sc[j] = exp(sc[j] - mx);
                    den += sc[j];
                }
                double* o = att + ((size_t)r * H + h) * hd;
                for (int i = 0; i < hd; ++i) o[i] = 0.0;
                for (int j = 0; j <= pos; ++j) {
                    const double* vj = kv->v + kv_index(dm, kv->cap, l, j, g);
                    double w = sc[j] / den;
                    for (int i = 0; i < hd; ++i) o[i] += w * vj[i];
                }
                free(sc);
            }
        }
        matmul_rows(M->bf16, Wl[W_O], d, H * hd, att, m, proj);
        for (size_t i = 0; i < (size_t)m * d; ++i) x[i] += proj[i];
        /* SwiGLU feed-forward sub-block */
        for (int r = 0; r < m; ++r) rmsnorm(M->bf16, Wl[W_FFN_NORM], d, dm->rms_eps, x + (size_t)r * d, nrm + (size_t)r * d);
        matmul_rows(M->bf16, Wl[W_GATE], F, d, nrm, m, gate);
        matmul_rows(M->bf16, Wl[W_UP], F, d, nrm, m, up);
        for (size_t i = 0; i < (size_t)m * F; ++i) {
            double u = up[i] + (ubias ? ubias[(size_t)l * F + i % F] : 0.0) + (cb ? cb[i] : 0.0);
            gate[i] = silu(gate[i]) * u;
        }
        matmul_rows(M->bf16, Wl[W_DOWN], d, F, gate, m, proj);
        for (size_t i = 0; i < (size_t)m * d; ++i) x[i] += proj[i] + (obias ? obias[i % d] : 0.0);
        if (taps) {
            int tl[3];
            tap_layers(dm->n_layers, tl);
            for (int sl = 0; sl < 3; ++sl)
                if (tl[sl] == l)
                    for (int r = 0; r < m; ++r)
                        memcpy(taps + ((size_t)r * 3 + sl) * d, x + (size_t)r * d, (size_t)d * sizeof(double));
        }
    }
    for (int r = 0; r < m; ++r) rmsnorm(M->bf16, M->final_norm, d, dm->rms_eps, x + (size_t)r * d, hF + (size_t)r * d);
    if (logits) matmul_rows(M->bf16, M->lm_head, dm->vocab, d, hF, m, logits);
    free(x); free(nrm); free(q); free(kk); free(vv); free(att); free(proj); free(gate); free(up);
    free(cb); free(ch);
}

/* ----------------------------------------------------------------------- */
/* Decisions, taken in float32                                              */
/* ----------------------------------------------------------------------- */

/* log sum_v exp(l_v / T) of a float32 logit row, rounded to float32. */
static float log_normaliser(const float* lg, int V, float T) {
    float mx = -INFINITY;
    for (int v = 0; v < V; ++v) {
        float s = lg[v] / T;
        if (s > mx) mx = s;
    }
    double acc = 0.0;
    for (int v = 0; v < V; ++v) acc += exp((double)(lg[v] / T - mx));
    return (float)((double)mx + log(acc));
}

/* argmax with ties to the lowest index; *margin = best - second best. */
static int argmax_margin(const float* sc, int V, float* margin) {
    int best = 0;
    for (int v = 1; v < V; ++v)
        if (sc[v] > sc[best]) best = v;
    float second = -INFINITY;
    for (int v = 0; v < V; ++v)
        if (v != best && sc[v] > second) second = sc[v];
    if (margin) *margin = sc[best] - second;
    return best;
}

/*
 * Draft pick from one drafter logit row (draft step j of the round that starts
 * at t, sequence b): Gumbel-max argmax_v(l_v/T + G_v) when T > 0, argmax when
 * T == 0.  *margin gets the gap between the two best scores.
 */
int oracle_pick(const float* q, int V, float T, uint64_t seed, int j, int t, int b, float* margin) {
    if (T == 0.0f) return argmax_margin(q, V, margin);
    float* sc = malloc((size_t)V * sizeof(float));
    for (int v = 0; v < V; ++v) sc[v] = q[v] / T + gumbel_at(seed, (uint32_t)v, (uint32_t)j, (uint32_t)t, PURPOSE_DRAFT, (uint32_t)b);
    int x = argmax_margin(sc, V, margin);
    free(sc);
    return x;
}

/* Per-round record of one sequence. */
typedef struct {
    int32_t active;            /* 0: sequence already finished, nothing done */
    int32_t t_start;
    int32_t n;                 /* accepted drafts */
    int32_t y;                 /* final token */
    int32_t count;             /* tokens emitted this round after truncation */
    int32_t used_fallback;     /* residual had no positive mass: drew from p */
    float final_margin;
    int32_t drafts[64];
    float draft_margin[64];
    float accept_margin[64];   /* |log u - log(p/q)|, or top-2 gap in greedy mode */
    float lse_v[65], lse_d[64];
} oround_log;

/*
 * Verification decisions for one block, given the k drafts, the verifier's
 * k+1 logit rows plog (row i scores the token after block input i) and the
 * drafter's k rows qlog (row i is the distribution draft i was drawn from).
 * T > 0: accept draft i iff log u_i < log p_i(x_i) - log q_i(x_i) (strict), u_i
 * a Philox uniform; n = leading accepts; the final token is a Gumbel-max draw
 * from (p_n - q_n)+ when n < k (from p_n if that residual has no positive
 * entry) and from p_k when n == k.  T == 0: accept iff the draft is the
 * verifier's argmax; final token = argmax of p_n.  Fills lg->n, lg->y and the
 * margins.
 */
void oracle_accept_final(int k, int V, float T, uint64_t seed, int t, int b, const int32_t* drafts,
                         const float* plog, const float* qlog, oround_log* lg) {
    int n = 0;
    float margin;
    if (T == 0.0f) {
        for (int i = 0; i < k; ++i) {
            int a = argmax_margin(plog + (size_t)i * V, V, &margin);
            lg->accept_margin[i] = margin;
            if (drafts[i] != a) break;
            ++n;
        }
        lg->n = n;
        lg->y = argmax_margin(plog + (size_t)n * V, V, &margin);
        lg->final_margin = margin;
        return;
    }
    float* sc = malloc((size_t)V * sizeof(float));
    for (int i = 0; i <= k; ++i) lg->lse_v[i] = log_normaliser(plog + (size_t)i * V, V, T);
    for (int i = 0; i < k; ++i) lg->lse_d[i] = log_normaliser(qlog + (size_t)i * V, V, T);
    for (int i = 0; i < k; ++i) {
        int x = drafts[i];
        float logp = plog[(size_t)i * V + x] / T - lg->lse_v[i];
        float logq = qlog[(size_t)i * V + x] / T - lg->lse_d[i];
        float ratio = logp - logq;
        float logu = logf(oracle_uniform(rng_word(seed, (uint32_t)i, 0, (uint32_t)t, PURPOSE_ACCEPT, (uint32_t)b, 0)));
        lg->accept_margin[i] = fabsf(logu - ratio);
        if (!(logu < ratio)) break;
        ++n;
    }
    const float* pr = plog + (size_t)n * V;
    int have_residual = 0;
    if (n < k) {
        const float* qr = qlog + (size_t)n * V;
        for (int v = 0; v < V; ++v) {
            float p = expf(pr[v] / T - lg->lse_v[n]);
            float q = expf(qr[v] / T - lg->lse_d[n]);
            float r = p - q;
            if (r > 0.0f) {
                sc[v] = logf(r) + gumbel_at(seed, (uint32_t)v, 0, (uint32_t)t, PURPOSE_FINAL, (uint32_t)b);
                have_residual = 1;
            } else {
                sc[v] = -INFINITY;
            }
        }
    }
    if (!have_residual) {
        for (int v = 0; v < V; ++v) sc[v] = pr[v] / T + gumbel_at(seed, (uint32_t)v, 0, (uint32_t)t, PURPOSE_FINAL, (uint32_t)b);
        lg->used_fallback = (n < k);
    }
    lg->n = n;
    lg->y = argmax_margin(sc, V, &margin);
    lg->final_margin = margin;
    free(sc);
}

/* ----------------------------------------------------------------------- */
/* Engine state                                                              */
/* ----------------------------------------------------------------------- */
typedef struct {
    omodel V, D;
    const void* w_s;           /* form 0: [d_D][d_V]; form 1: [L_D*F_D][d_V]; storage type of the models */
    int form;                  /* 0: input-embedding steering; 1: MLP steering (eq. (2)); 2: bias after the MLP;
                                  3: conditional bias in the MLP */
    const void *w_cf, *w_cu;   /* form 3: V^f [L_D*R][d_D], U [L_D*F_D][R]; W_s holds V^g [L_D*R][d_V] */
    int rank;                  /* form 3: R */
    const void *w_hml, *ln_gain, *ln_bias;   /* form 1: W_hml [d_V][3 d_V], LayerNorm gain and shift [d_V] */
    double ln_eps;
    double* ub;                /* form 1: [max_batch][L_D*F_D] up-projection biases; form 2: [max_batch][d_D];
                                  form 3: [max_batch][L_D*R] the g parts V_l^g g */
    int nb;                    /* bias values per sequence */
    int k, max_batch, cap, max_new;
    float temperature;
    uint64_t seed;
    /* per sequence */
    int batch;
    int32_t* hist;             /* [max_batch][cap] */
    int32_t *t, *len_v, *len_d, *produced, *done;
    double* s;                 /* [max_batch][d_D] */
    okv *kv_v, *kv_d;
    int prefilled;
} ostate;

static okv kv_alloc(const odims* dm, int cap) {
    okv kv;
    kv.cap = cap;
    size_t n = (size_t)dm->n_layers * cap * dm->n_kv_heads * (dm->d_model / dm->n_heads);
    kv.k = calloc(n, sizeof(double));
    kv.v = calloc(n, sizeof(double));
    return kv;
}

ostate* oracle_create(const int32_t* dims_v, const double* rope_eps_v, const int32_t* dims_d,
                      const double* rope_eps_d, int bf16, const void* const* ptrs_v, const void* const* ptrs_d,
                      const void* w_s, int k, int max_batch, int cap, int max_new, float temperature,
                      uint64_t seed, int form, const void* w_hml, const void* ln_gain, const void* ln_bias,
                      double ln_eps, const void* w_cf, const void* w_cu, int rank) {
    /* MLP steering taps decoder block 3: the verifier needs at least three layers */
    if (form != 0 && ((form < 1 || form > 3) || dims_v[0] < 3 || !w_hml || !ln_gain || !ln_bias)) return NULL;
    if (form == 3 && (!w_cf || !w_cu || rank < 1)) return NULL;
    ostate* st = calloc(1, sizeof(ostate));
    omodel* ms[2] = {&st->V, &st->D};
    const int32_t* dims[2] = {dims_v, dims_d};
    const double* re[2] = {rope_eps_v, rope_eps_d};
    const void* const* ptrs[2] = {ptrs_v, ptrs_d};
    for (int i = 0; i < 2; ++i) {
        omodel* M = ms[i];
        M->dm.n_layers = dims[i][0]; M->dm.d_model = dims[i][1]; M->dm.n_heads = dims[i][2];
        M->dm.n_kv_heads = dims[i][3]; M->dm.d_ff = dims[i][4]; M->dm.vocab = dims[i][5];
        M->dm.rope_theta = re[i][0]; M->dm.rms_eps = re[i][1];
        M->bf16 = bf16;
        /* pointer list: embed, n_layers*9 layer tensors, final_norm, lm_head */
        M->embed = ptrs[i][0];
        M->layers = (const void**)(ptrs[i] + 1);
        M->final_norm = ptrs[i][1 + (size_t)M->dm.n_layers * W_PER_LAYER];
        M->lm_head = ptrs[i][2 + (size_t)M->dm.n_layers * W_PER_LAYER];
    }
    st->w_s = w_s;
    st->form = form;
    st->w_hml = w_hml; st->ln_gain = ln_gain; st->ln_bias = ln_bias; st->ln_eps = ln_eps;
    st->w_cf = w_cf; st->w_cu = w_cu; st->rank = rank;
    st->nb = form == 1 ? st->D.dm.n_layers * st->D.dm.d_ff
           : form == 2 ? st->D.dm.d_model
           : form == 3 ? st->D.dm.n_layers * rank : 0;
    if (form != 0) st->ub = calloc((size_t)max_batch * st->nb, sizeof(double));
    st->k = k; st->max_batch = max_batch; st->cap = cap; st->max_new = max_new;
    st->temperature = temperature; st->seed = seed;
    st->hist = calloc((size_t)max_batch * cap, sizeof(int32_t));
    st->t = calloc(max_batch, sizeof(int32_t));
    st->len_v = calloc(max_batch, sizeof(int32_t));
    st->len_d = calloc(max_batch, sizeof(int32_t));
    st->produced = calloc(max_batch, sizeof(int32_t));
    st->done = calloc(max_batch, sizeof(int32_t));
    st->s = calloc((size_t)max_batch * st->D.dm.d_model, sizeof(double));
    st->kv_v = calloc(max_batch, sizeof(okv));
    st->kv_d = calloc(max_batch, sizeof(okv));
    return st;
}

void oracle_destroy(ostate* st) {
    if (!st) return;
    for (int b = 0; b < st->max_batch; ++b) {
        free(st->kv_v[b].k); free(st->kv_v[b].v);
        free(st->kv_d[b].k); free(st->kv_d[b].v);
    }
    free(st->kv_v); free(st->kv_d);
    free(st->hist); free(st->t); free(st->len_v); free(st->len_d); free(st->produced); free(st->done);
    free(st->s);
    free(st->ub);
    free(st);
}

/* s = W_s h  (W_s is [d_D][d_V]) */
static void steer(const ostate* st, const double* h, double* s) {
    matmul_rows(st->V.bf16, st->w_s, st->D.dm.d_model, st->V.dm.d_model, h, 1, s);
}

/* MLP steering (eq. (2)): g = LayerNorm(W_hml [h; m; l]), then the biases
 * ub = W_s g: per-layer up-projection biases [L_D*F_D] (form 1), the one
 * bias after every MLP [d_D] (form 2), or the g parts V_l^g g of the
 * conditional biases [L_D*R] (form 3).  z holds [h; m; l] (3 d_V). */
static void mlp_steer(const ostate* st, const double* z, double* ub) {
    int dV = st->V.dm.d_model;
    int nb = st->nb;
    double* g = malloc((size_t)dV * sizeof(double));
    matmul_rows(st->V.bf16, st->w_hml, dV, 3 * dV, z, 1, g);
    double mean = 0.0;
    for (int i = 0; i < dV; ++i) mean += g[i];
    mean /= dV;
    double var = 0.0;
    for (int i = 0; i < dV; ++i) var += (g[i] - mean) * (g[i] - mean);
    var /= dV;
    double inv = 1.0 / sqrt(var + st->ln_eps);
    for (int i = 0; i < dV; ++i)
        g[i] = (g[i] - mean) * inv * wval(st->V.bf16, st->ln_gain, i) + wval(st->V.bf16, st->ln_bias, i);
    matmul_rows(st->V.bf16, st->w_s, nb, dV, g, 1, ub);
    free(g);
}

/*
 * Prefill sequence slot b with prompt x_0..x_{p-1}: both models process
 * x_0..x_{p-2}; the drafter does so with zero steering; the steering vector
 * for the first round is W_s applied to the verifier's final-norm hidden state
 * at position p-2 (zero when p == 1).  Afterwards t = p and both caches hold
 * p-1 positions.  Returns 0, or -1 on bad arguments.
 */
int oracle_prefill_one(ostate* st, int b, const int32_t* prompt, int p) {
    if (b < 0 || b >= st->max_batch || p < 1 || p + st->max_new + st->k + 1 > st->cap) return -1;
    if (!st->kv_v[b].k) {
        st->kv_v[b] = kv_alloc(&st->V.dm, st->cap);
        st->kv_d[b] = kv_alloc(&st->D.dm, st->cap);
    }
    int dV = st->V.dm.d_model, dD = st->D.dm.d_model;
    memcpy(st->hist + (size_t)b * st->cap, prompt, (size_t)p * sizeof(int32_t));
    double* s = st->s + (size_t)b * dD;
    for (int i = 0; i < dD; ++i) s[i] = 0.0;
    size_t nb = (size_t)st->nb;
    double* ub = st->form != 0 ? st->ub + (size_t)b * nb : NULL;
    if (ub)
        for (size_t i = 0; i < nb; ++i) ub[i] = 0.0;
    if (p >= 2) {
        double* hF = malloc((size_t)(p - 1) * dV * sizeof(double));
        double* taps = ub ? malloc((size_t)(p - 1) * 3 * dV * sizeof(double)) : NULL;
        forward_block(&st->V, &st->kv_v[b], 0, p - 1, prompt, NULL, NULL, NULL, NULL, taps, hF, NULL);
        if (ub) mlp_steer(st, taps + (size_t)(p - 2) * 3 * dV, ub);
        else steer(st, hF + (size_t)(p - 2) * dV, s);
        free(hF);
        free(taps);
        /* the drafter processes the prompt without steering */
        double* hD = malloc((size_t)(p - 1) * dD * sizeof(double));
        forward_block(&st->D, &st->kv_d[b], 0, p - 1, prompt, NULL, NULL, NULL, NULL, NULL, hD, NULL);
        free(hD);
    }
    st->t[b] = p;
    st->len_v[b] = p - 1;
    st->len_d[b] = p - 1;
    st->produced[b] = 0;
    st->done[b] = 0;
    if (b + 1 > st->batch) st->batch = b + 1;
    st->prefilled = 1;
    return 0;
}


/*
 * One speculative round for sequence b.  Optional dumps: logits_v [k+1][V],
 * logits_d [k][V] (float32 as used by the decisions), hf_v [k+1][d_V] (double).
 * Writes the emitted tokens to out_tokens[0..count-1].
 */
int oracle_round_one(ostate* st, int b, int32_t* out_tokens, oround_log* lg, float* logits_v_dump,
                     float* logits_d_dump, double* hf_v_dump) {
    memset(lg, 0, sizeof(*lg));
    if (!st->prefilled || b < 0 || b >= st->batch) return -1;
    if (st->done[b]) return 0;
    int k = st->k, V = st->V.dm.vocab, dV = st->V.dm.d_model, dD = st->D.dm.d_model;
    float T = st->temperature;
    int32_t* hist = st->hist + (size_t)b * st->cap;
    int t = st->t[b];
    double* s = st->s + (size_t)b * dD;
    double* ub = st->form != 0 ? st->ub + (size_t)b * st->nb : NULL;
    lg->active = 1;
    lg->t_start = t;

    float* qlog = malloc((size_t)k * V * sizeof(float));   /* drafter logits rows q_1..q_k */
    float* plog = malloc((size_t)(k + 1) * V * sizeof(float));
    double* dl = malloc((size_t)2 * V * sizeof(double));
    double* hD = malloc((size_t)2 * dD * sizeof(double));
    int32_t drafts[64];

    /* ---- drafting: catch-up tokens, then k-1 single-token steps ---- */
    for (int j = 1; j <= k; ++j) {
        int pos0, m;
        const int32_t* in;
        if (j == 1) {
            pos0 = st->len_d[b];
            m = t - pos0;                 /* 1 or 2 catch-up tokens */
            in = hist + pos0;
        } else {
            pos0 = t + j - 2;
            m = 1;
            in = &drafts[j - 2];
        }
        ocond cd = {st->w_cf, st->w_cu, st->rank, ub};
        forward_block(&st->D, &st->kv_d[b], pos0, m, in, ub ? NULL : s, st->form == 1 ? ub : NULL,
                      st->form == 2 ? ub : NULL, st->form == 3 ? &cd : NULL, NULL, hD, dl);
        float* q = qlog + (size_t)(j - 1) * V;
        for (int v = 0; v < V; ++v) q[v] = (float)dl[(size_t)(m - 1) * V + v];
        float margin;
        drafts[j - 1] = oracle_pick(q, V, T, st->seed, j, t, b, &margin);
        lg->drafts[j - 1] = drafts[j - 1];
        lg->draft_margin[j - 1] = margin;
    }

    /* ---- verification of the block [x_{t-1}, drafts] at positions t-1..t+k-1 ---- */
    int32_t blk[65];
    blk[0] = hist[t - 1];
    for (int i = 0; i < k; ++i) blk[i + 1] = drafts[i];
    double* hF = malloc((size_t)(k + 1) * dV * sizeof(double));
    double* vl = malloc((size_t)(k + 1) * V * sizeof(double));
    double* taps = ub ? malloc((size_t)(k + 1) * 3 * dV * sizeof(double)) : NULL;
    forward_block(&st->V, &st->kv_v[b], t - 1, k + 1, blk, NULL, NULL, NULL, NULL, taps, hF, vl);
    for (size_t i = 0; i < (size_t)(k + 1) * V; ++i) plog[i] = (float)vl[i];

    /* ---- accept / reject, final token ---- */
    oracle_accept_final(k, V, T, st->seed, t, b, drafts, plog, qlog, lg);
    int n = lg->n;

    /* ---- commit: emit accepted drafts + final token, roll back KV lengths ---- */
    int remaining = st->max_new - st->produced[b];
    int count = n + 1 < remaining ? n + 1 : remaining;
    for (int i = 0; i < n; ++i) hist[t + i] = drafts[i];
    hist[t + n] = lg->y;
    for (int i = 0; i < count; ++i) out_tokens[i] = hist[t + i];
    lg->count = count;
    st->produced[b] += count;
    if (st->produced[b] >= st->max_new) st->done[b] = 1;
    st->len_v[b] = t + n;
    st->len_d[b] = (t + k - 1 < t + n) ? t + k - 1 : t + n;
    st->t[b] = t + n + 1;
    if (ub) mlp_steer(st, taps + (size_t)n * 3 * dV, ub);
    else steer(st, hF + (size_t)n * dV, s);

    if (logits_v_dump) memcpy(logits_v_dump, plog, (size_t)(k + 1) * V * sizeof(float));
    if (logits_d_dump) memcpy(logits_d_dump, qlog, (size_t)k * V * sizeof(float));
    if (hf_v_dump) memcpy(hf_v_dump, hF, (size_t)(k + 1) * dV * sizeof(double));
    for (int i = 0; i < k; ++i) lg->drafts[i] = drafts[i];
    free(qlog); free(plog); free(dl); free(hD); free(hF); free(vl); free(taps);
    return 0;
}

/* ----------------------------------------------------------------------- */
/* Accessors used by the tests                                               */
/* ----------------------------------------------------------------------- */
void oracle_get_state(const ostate* st, int b, int32_t* t, int32_t* len_v, int32_t* len_d, int32_t* produced,
                      int32_t* done) {
    *t = st->t[b]; *len_v = st->len_v[b]; *len_d = st->len_d[b];
    *produced = st->produced[b]; *done = st->done[b];
}

void oracle_get_steer(const ostate* st, int b, double* out) {
    memcpy(out, st->s + (size_t)b * st->D.dm.d_model, (size_t)st->D.dm.d_model * sizeof(double));
}

void oracle_set_steer(ostate* st, int b, const double* in) {
    memcpy(st->s + (size_t)b * st->D.dm.d_model, in, (size_t)st->D.dm.d_model * sizeof(double));
}

/* Forms 1 and 2: the biases of sequence b for its next round ([L_D*F_D] or [d_D]). */
void oracle_get_ubias(const ostate* st, int b, double* out) {
    memcpy(out, st->ub + (size_t)b * st->nb, (size_t)st->nb * sizeof(double));
}

void oracle_get_hist(const ostate* st, int b, int32_t* out, int n) {
    memcpy(out, st->hist + (size_t)b * st->cap, (size_t)n * sizeof(int32_t));
}

int oracle_round_log_size(void) { return (int)sizeof(oround_log); }

void oracle_set_seed(ostate* st, uint64_t seed) { st->seed = seed; }

/*
 * Stand-alone forward of a whole sequence from an empty cache: one model
 * (0 = verifier, 1 = drafter), tokens x_0..x_{n-1}, optional per-position
 * additive input vectors add[n][d] (NULL for none).  Outputs final-norm hidden
 * states [n][d] and logits [n][vocab] in double.
 */
void oracle_forward(const ostate* st, int which, const int32_t* toks, int n, const double* add, double* hF,
                    double* logits) {
    const omodel* M = which == 0 ? &st->V : &st->D;
    okv kv = kv_alloc(&M->dm, n);
    if (!add) {
        forward_block(M, &kv, 0, n, toks, NULL, NULL, NULL, NULL, NULL, hF, logits);
    } else {
        int d = M->dm.d_model;
        for (int i = 0; i < n; ++i)
            forward_block(M, &kv, i, 1, toks + i, add + (size_t)i * d, NULL, NULL, NULL, NULL, hF + (size_t)i * d,
                          logits ? logits + (size_t)i * M->dm.vocab : NULL);
    }
    free(kv.k);
    free(kv.v);
}

/* Steering projection on its own: s = W_s h. */
void oracle_steer(const ostate* st, const double* h, double* s) { steer(st, h, s); }

/*
 * Whole-sequence forward with the MLP-steering pieces exposed: optional
 * per-layer up-projection biases ubias[L][d_ff] and a bias after every MLP
 * obias[d] (NULL for none) applied to every row, and the three steering taps
 * of every row, taps[n][3][d] (NULL for none).  Outputs as oracle_forward.
 */
void oracle_forward_mlp(const ostate* st, int which, const int32_t* toks, int n, const double* ubias,
                        const double* obias, double* taps, double* hF, double* logits) {
    const omodel* M = which == 0 ? &st->V : &st->D;
    okv kv = kv_alloc(&M->dm, n);
    forward_block(M, &kv, 0, n, toks, NULL, ubias, obias, NULL, taps, hF, logits);
    free(kv.k);
    free(kv.v);
}

/* MLP steering on its own: ub = W_s LayerNorm(W_hml z), z = [h; m; l] (form 1 or 2 sizes). */
void oracle_mlp_steer(const ostate* st, const double* z, double* ub) { mlp_steer(st, z, ub); }

/*
 * Whole-sequence forward of the drafter (which = 1) or verifier with the conditional MLP bias of
 * form 3 on every row: c [L*R] holds V_l^g g for one g (NULL: no bias).  Outputs as oracle_forward.
 */
void oracle_forward_cond(const ostate* st, int which, const int32_t* toks, int n, const double* c, double* hF,
                         double* logits) {
    const omodel* M = which == 0 ? &st->V : &st->D;
    okv kv = kv_alloc(&M->dm, n);
    ocond cd = {st->w_cf, st->w_cu, st->rank, c};
    forward_block(M, &kv, 0, n, toks, NULL, NULL, NULL, c ? &cd : NULL, NULL, hF, logits);
    free(kv.k);
    free(kv.v);
}

/*
 * Training-objective forward (input-form steering) over tokens x_0..x_{n-1}: deltas[tau] in 1..k
 * is the offset of target tau (deltas[0] unused).  out_kl[tau] (tau = 1..n-1) receives
 *   KL(p_V || p_D) = sum_v p_V(v) (log p_V(v) - log p_D(v)),
 * p_V = softmax of the verifier's logits at position tau-1 and p_D = softmax of the drafter's
 * logits at position tau-1, where the drafter's input embedding at every position p is
 * E_D[x_p] + s_{p+1}, s_tau = W_s hF_V(tau - deltas[tau] - 1) (zero when that position is
 * negative), hF_V(q) the verifier's final-norm hidden state at position q.  out_kl[0] = 0.
 * out_spread (NULL for none) receives sum_v p_V(v) |d_v - E_pV[d]| with d = log p_V - log p_D, the
 * sensitivity of KL to errors in the verifier's logits.  Returns the mean of out_kl[1..n-1]; NaN
 * for n < 2.
 */
double oracle_train_loss(const ostate* st, const int32_t* toks, int n, const int32_t* deltas, double* out_kl,
                         double* out_spread) {
    if (n < 2) return NAN;
    int dV = st->V.dm.d_model, dD = st->D.dm.d_model, V = st->V.dm.vocab, m = n - 1;
    double* hF = malloc((size_t)m * dV * sizeof(double));
    double* lv = malloc((size_t)m * V * sizeof(double));
    double* hD = malloc((size_t)dD * sizeof(double));
    double* ld = malloc((size_t)m * V * sizeof(double));
    double* sv = malloc((size_t)dD * sizeof(double));
    okv kvv = kv_alloc(&st->V.dm, m), kvd = kv_alloc(&st->D.dm, m);
    /* verifier over x_0..x_{n-2}: hidden states and logits of every position */
    forward_block(&st->V, &kvv, 0, m, toks, NULL, NULL, NULL, NULL, NULL, hF, lv);
    /* drafter one position at a time, each with the steering of the target it predicts */
    for (int p = 0; p < m; ++p) {
        int q = p - deltas[p + 1];
        if (q >= 0) steer(st, hF + (size_t)q * dV, sv);
        else
            for (int i = 0; i < dD; ++i) sv[i] = 0.0;
        forward_block(&st->D, &kvd, p, 1, toks + p, sv, NULL, NULL, NULL, NULL, hD, ld + (size_t)p * V);
    }
    double sum = 0.0;
    out_kl[0] = 0.0;
    for (int p = 0; p < m; ++p) {
        const double* a = lv + (size_t)p * V;
        const double* b = ld + (size_t)p * V;
        double ma = -INFINITY, mb = -INFINITY;
        for (int v = 0; v < V; ++v) {
            if (a[v] > ma) ma = a[v];
            if (b[v] > mb) mb = b[v];
        }
        double za = 0.0, zb = 0.0;
        for (int v = 0; v < V; ++v) {
            za += exp(a[v] - ma);
            zb += exp(b[v] - mb);
        }
        double lsa = ma + log(za), lsb = mb + log(zb), kl = 0.0;
        for (int v = 0; v < V; ++v) {
            double lpa = a[v] - lsa, lpb = b[v] - lsb;
            kl += exp(lpa) * (lpa - lpb);
        }
        out_kl[p + 1] = kl;
        if (out_spread) {
            double spread = 0.0;
            for (int v = 0; v < V; ++v) spread += exp(a[v] - lsa) * fabs((a[v] - lsa) - (b[v] - lsb) - kl);
            out_spread[p + 1] = spread;
        }
        sum += kl;
    }
    free(hF); free(lv); free(hD); free(ld); free(sv);
    free(kvv.k); free(kvv.v); free(kvd.k); free(kvd.v);
    return sum / m;
}
