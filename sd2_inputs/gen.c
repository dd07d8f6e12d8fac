/*
 * Seeded synthetic inputs shared by the CPU oracle and the GPU path.
 *
 * This module holds none of the speculative-decoding arithmetic: it only turns
 * (seed, purpose, tensor id, index) into weight values and prompt token ids.
 *
 *  - Counter-based generator: Philox4x32-10 as defined by Salmon, Moraes, Dror
 *    and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11).  This is
 *    the generator module's own copy; the oracle and the GPU sampler each carry
 *    an independent implementation of their own.
 *  - Normal variates: the Box-Muller transform in float64 on two 53-bit uniforms
 *    taken from one Philox block; element i uses the cosine (even i) or the sine
 *    (odd i) branch of block i/2.  The value scale*z is rounded to float32
 *    (round-to-nearest-even) and, for bf16 tensors, from float32 to bf16 (RNE).
 *  - Prompt ids: Lemire's multiply-shift map of one 32-bit word onto [0, V).
 *
 * Counter layout: (c0, c1) = 64-bit element/pair index, c2 = tensor or sequence
 * id, c3 = purpose << 24.  Key = (seed low word, seed high word).
 */
#include <stdint.h>
#include <math.h>
#include <string.h>

#define GEN_PURPOSE_WEIGHT 0x10u
#define GEN_PURPOSE_PROMPT 0x11u
#define GEN_PURPOSE_PROMPT_LEN 0x12u

static void gen_philox(const uint32_t ctr_in[4], uint64_t seed, uint32_t out[4]) {
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int r = 0; r < 10; ++r) {
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

/* Normal pair for block j of tensor `tensor_id`. */
static void normal_pair(uint64_t seed, uint32_t tensor_id, uint64_t j, double* z0, double* z1) {
    uint32_t ctr[4] = {(uint32_t)j, (uint32_t)(j >> 32), tensor_id, GEN_PURPOSE_WEIGHT << 24};
    uint32_t w[4];
    gen_philox(ctr, seed, w);
    uint64_t a = ((uint64_t)w[1] << 32) | w[0];
    uint64_t b = ((uint64_t)w[3] << 32) | w[2];
    double u1 = ((double)(a >> 11) + 0.5) * (1.0 / 9007199254740992.0); /* (0,1) */
    double u2 = ((double)(b >> 11) + 0.5) * (1.0 / 9007199254740992.0);
    double r = sqrt(-2.0 * log(u1));
    double th = 6.283185307179586476925286766559 * u2;
    *z0 = r * cos(th);
    *z1 = r * sin(th);
}

/* out[i] = RNE_bf16(RNE_f32(scale * z_i)), i in [0, n). */
void gen_normal_bf16(uint16_t* out, uint64_t n, uint64_t seed, uint32_t tensor_id, double scale) {
    int64_t npairs = (int64_t)((n + 1) / 2);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < npairs; ++j) {
        double z0, z1;
        normal_pair(seed, tensor_id, (uint64_t)j, &z0, &z1);
        uint64_t i = (uint64_t)j * 2;
        out[i] = f32_to_bf16_rne((float)(scale * z0));
        if (i + 1 < n) out[i + 1] = f32_to_bf16_rne((float)(scale * z1));
    }
}

/* out[i] = RNE_f32(scale * z_i). */
void gen_normal_f32(float* out, uint64_t n, uint64_t seed, uint32_t tensor_id, double scale) {
    int64_t npairs = (int64_t)((n + 1) / 2);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < npairs; ++j) {
        double z0, z1;
        normal_pair(seed, tensor_id, (uint64_t)j, &z0, &z1);
        uint64_t i = (uint64_t)j * 2;
        out[i] = (float)(scale * z0);
        if (i + 1 < n) out[i + 1] = (float)(scale * z1);
    }
}

/* Uniform integers in [lo, hi] (inclusive) for purpose/stream; one Philox block per value. */
void gen_uniform_int(int32_t* out, uint64_t n, uint64_t seed, uint32_t purpose, uint32_t stream,
                     int32_t lo, int32_t hi) {
    uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), stream, purpose << 24};
        uint32_t w[4];
        gen_philox(ctr, seed, w);
        out[i] = lo + (int32_t)(((uint64_t)w[0] * span) >> 32);
    }
}

/* Prompt ids for sequence b: n ids uniform in [0, vocab). */
void gen_prompt(int32_t* out, uint64_t n, uint64_t seed, uint32_t b, int32_t vocab) {
    gen_uniform_int(out, n, seed, GEN_PURPOSE_PROMPT, b, 0, vocab - 1);
}

/* Per-sequence prompt lengths uniform in [lo, hi]. */
void gen_prompt_lens(int32_t* out, uint64_t n, uint64_t seed, int32_t lo, int32_t hi) {
    gen_uniform_int(out, n, seed, GEN_PURPOSE_PROMPT_LEN, 0, lo, hi);
}

/* Raw block, exposed so a test can check the generator's Philox on its own. */
void gen_philox_block(const uint32_t ctr[4], uint64_t seed, uint32_t out[4]) { gen_philox(ctr, seed, out); }
