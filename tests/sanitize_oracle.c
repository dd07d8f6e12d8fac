/*
 * Driver for the oracle under AddressSanitizer and UndefinedBehaviorSanitizer (test
 * infrastructure, built and run by tests/test_oracle_sanitizers.py; CPU only).
 *
 * A tiny verifier (3 layers, so that the MLP steering taps exist) and drafter, with weights from
 * a fixed linear congruential generator, in float32 and in bf16 storage; for every steering form
 * (input, MLP, bias after the MLP, conditional bias) it prefills two sequences of different
 * prompt lengths, runs rounds until both are done, and calls the whole-sequence forward and, for
 * the input form, the training-objective forward.  Exit status 0 when every call returned what
 * it should; the sanitizers abort on the first error they find.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct ostate ostate;
ostate* oracle_create(const int32_t* dims_v, const double* rope_eps_v, const int32_t* dims_d,
                      const double* rope_eps_d, int bf16, const void* const* ptrs_v, const void* const* ptrs_d,
                      const void* w_s, int k, int max_batch, int cap, int max_new, float temperature,
                      uint64_t seed, int form, const void* w_hml, const void* ln_gain, const void* ln_bias,
                      double ln_eps, const void* w_cf, const void* w_cu, int rank);
void oracle_destroy(ostate* st);
int oracle_prefill_one(ostate* st, int b, const int32_t* prompt, int p);
int oracle_round_one(ostate* st, int b, int32_t* out_tokens, void* lg, float* logits_v_dump,
                     float* logits_d_dump, double* hf_v_dump);
int oracle_round_log_size(void);
void oracle_get_state(const ostate* st, int b, int32_t* t, int32_t* len_v, int32_t* len_d, int32_t* produced,
                      int32_t* done);
void oracle_forward(const ostate* st, int which, const int32_t* toks, int n, const double* add, double* hF,
                    double* logits);
double oracle_train_loss(const ostate* st, const int32_t* toks, int n, const int32_t* deltas, double* out_kl,
                         double* out_spread);

static uint64_t lcg = 0x9e3779b97f4a7c15ull;
static double next_val(double scale) {
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    return scale * ((double)(lcg >> 11) / 9007199254740992.0 - 0.5);
}

/* one tensor of n values, float32 or bf16 (round to nearest even); gains are ones */
static void* tensor(int bf16, size_t n, double scale, int ones) {
    if (bf16) {
        uint16_t* p = malloc(n * sizeof(uint16_t));
        for (size_t i = 0; i < n; ++i) {
            float f = ones ? 1.0f : (float)next_val(scale);
            uint32_t u;
            memcpy(&u, &f, 4);
            u += 0x7fffu + ((u >> 16) & 1u);
            p[i] = (uint16_t)(u >> 16);
        }
        return p;
    }
    float* p = malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = ones ? 1.0f : (float)next_val(scale);
    return p;
}

/* pointer list: embed, per layer (attn norm, Wq, Wk, Wv, Wo, ffn norm, gate, up, down), final norm, LM head */
static void** model(int bf16, const int32_t* d) {
    int L = d[0], dm = d[1], H = d[2], Hkv = d[3], F = d[4], V = d[5], hd = dm / H;
    void** p = malloc(sizeof(void*) * (size_t)(3 + 9 * L));
    p[0] = tensor(bf16, (size_t)V * dm, 0.5, 0);
    for (int l = 0; l < L; ++l) {
        void** w = p + 1 + 9 * l;
        w[0] = tensor(bf16, dm, 0, 1);
        w[1] = tensor(bf16, (size_t)H * hd * dm, 0.3, 0);
        w[2] = tensor(bf16, (size_t)Hkv * hd * dm, 0.3, 0);
        w[3] = tensor(bf16, (size_t)Hkv * hd * dm, 0.3, 0);
        w[4] = tensor(bf16, (size_t)dm * H * hd, 0.3, 0);
        w[5] = tensor(bf16, dm, 0, 1);
        w[6] = tensor(bf16, (size_t)F * dm, 0.3, 0);
        w[7] = tensor(bf16, (size_t)F * dm, 0.3, 0);
        w[8] = tensor(bf16, (size_t)dm * F, 0.3, 0);
    }
    p[1 + 9 * L] = tensor(bf16, dm, 0, 1);
    p[2 + 9 * L] = tensor(bf16, (size_t)V * dm, 0.3, 0);
    return p;
}

static void free_model(void** p, int L) {
    for (int i = 0; i < 3 + 9 * L; ++i) free(p[i]);
    free(p);
}

static int run(int bf16, int form) {
    const int32_t dv[6] = {3, 64, 4, 2, 128, 96}, dd[6] = {2, 32, 2, 1, 64, 96};
    const double re[2] = {1e4, 1e-5};
    const int k = 3, B = 2, cap = 64, max_new = 12, R = 8;
    void** mv = model(bf16, dv);
    void** md = model(bf16, dd);
    void *ws = NULL, *hml = NULL, *g = NULL, *bsh = NULL, *cf = NULL, *cu = NULL;
    if (form == 0) ws = tensor(bf16, (size_t)dd[1] * dv[1], 0.3, 0);
    if (form == 1) ws = tensor(bf16, (size_t)dd[0] * dd[4] * dv[1], 0.3, 0);
    if (form == 2) ws = tensor(bf16, (size_t)dd[1] * dv[1], 0.3, 0);
    if (form == 3) {
        ws = tensor(bf16, (size_t)dd[0] * R * dv[1], 0.3, 0);
        cf = tensor(bf16, (size_t)dd[0] * R * dd[1], 0.3, 0);
        cu = tensor(bf16, (size_t)dd[0] * dd[4] * R, 0.3, 0);
    }
    if (form != 0) {
        hml = tensor(bf16, (size_t)dv[1] * 3 * dv[1], 0.3, 0);
        g = tensor(bf16, dv[1], 0, 1);
        bsh = tensor(bf16, dv[1], 0.1, 0);
    }
    ostate* st = oracle_create(dv, re, dd, re, bf16, (const void* const*)mv, (const void* const*)md, ws, k, B,
                               cap, max_new, 1.0f, 7, form, hml, g, bsh, 1e-5, cf, cu, form == 3 ? R : 0);
    int bad = 0;
    if (!st) {
        fprintf(stderr, "oracle_create failed (bf16 %d, form %d)\n", bf16, form);
        return 1;
    }
    const int32_t prompt0[5] = {3, 17, 42, 5, 90}, prompt1[1] = {11};
    bad |= oracle_prefill_one(st, 0, prompt0, 5) != 0;
    bad |= oracle_prefill_one(st, 1, prompt1, 1) != 0;
    void* lg = malloc((size_t)oracle_round_log_size());
    float* lv = malloc(sizeof(float) * (size_t)(k + 1) * dv[5]);
    float* ld = malloc(sizeof(float) * (size_t)k * dd[5]);
    double* hv = malloc(sizeof(double) * (size_t)(k + 1) * dv[1]);
    int32_t out[16];
    for (int r = 0; r < 64; ++r) {
        int live = 0;
        for (int b = 0; b < B; ++b) {
            int32_t t, lvn, ldn, produced, done;
            oracle_get_state(st, b, &t, &lvn, &ldn, &produced, &done);
            if (done) continue;
            live = 1;
            if (oracle_round_one(st, b, out, lg, lv, ld, hv) < 0) bad = 1;
        }
        if (!live) break;
    }
    for (int b = 0; b < B; ++b) {
        int32_t t, lvn, ldn, produced, done;
        oracle_get_state(st, b, &t, &lvn, &ldn, &produced, &done);
        if (!done || produced != max_new) bad = 1;
    }
    const int n = 9;
    const int32_t toks[9] = {1, 2, 3, 4, 5, 6, 7, 8, 9};
    double* hF = malloc(sizeof(double) * (size_t)n * dv[1]);
    double* lgt = malloc(sizeof(double) * (size_t)n * dv[5]);
    oracle_forward(st, 0, toks, n, NULL, hF, lgt);
    oracle_forward(st, 1, toks, n, NULL, hF, lgt);
    if (form == 0) {
        const int32_t deltas[9] = {0, 1, 2, 3, 1, 2, 3, 1, 2};
        double kl[9], spread[9];
        const double mean = oracle_train_loss(st, toks, n, deltas, kl, spread);
        if (!(mean >= 0.0) || !isfinite(mean)) bad = 1;
    }
    free(hF); free(lgt); free(lg); free(lv); free(ld); free(hv);
    oracle_destroy(st);
    free_model(mv, dv[0]);
    free_model(md, dd[0]);
    free(ws); free(hml); free(g); free(bsh); free(cf); free(cu);
    if (bad) fprintf(stderr, "unexpected result (bf16 %d, form %d)\n", bf16, form);
    return bad;
}

int main(void) {
    int bad = 0;
    for (int bf16 = 0; bf16 < 2; ++bf16)
        for (int form = 0; form < 4; ++form) bad |= run(bf16, form);
    if (!bad) printf("oracle sanitizer run: 8 configurations clean\n");
    return bad;
}
