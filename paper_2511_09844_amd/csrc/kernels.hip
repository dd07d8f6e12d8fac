// SD^2 round kernels for gfx950: input planning, weight-streaming GEMV, RoPE/KV append,
// grouped-query attention, and the vocabulary-wide sampler.
#include <math.h>

#include "device_common.h"
#include "engine.h"

namespace sd2 {

// ===========================================================================
// RoPE table: cos/sin(pos * theta^(-2i/hd)) evaluated in double, stored as float.
// ===========================================================================
__global__ void k_rope_table(float* __restrict__ c, float* __restrict__ s, int cap, int half, int hd, double theta) {
    int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= cap * half) return;
    int pos = idx / half, i = idx % half;
    double ang = (double)pos * pow(theta, -2.0 * (double)i / (double)hd);
    c[idx] = (float)cos(ang);
    s[idx] = (float)sin(ang);
}

void launch_rope_table(hipStream_t s, ModelDev& m, int cap) {
    int half = m.hd / 2;
    int n = cap * half;
    k_rope_table<<<(n + 255) / 256, 256, 0, s>>>(m.rope_cos, m.rope_sin, cap, half, m.hd, (double)m.dm.rope_theta);
}

// Static drafter LM-head output maps: step 1 has two rows per sequence (catch-up), of which
// only the second (position t-1) produces logits; later steps have one row per sequence.
__global__ void k_init_maps(int32_t* lm_map_d, int32_t* ident, int max_batch, int k) {
    int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < 2 * max_batch) ident[r] = r;
    for (int j = 0; j < k; ++j) {
        int32_t* mp = lm_map_d + (size_t)j * 2 * max_batch;
        if (j == 0) {
            if (r < 2 * max_batch) mp[r] = (r & 1) ? (r >> 1) * k : -1;
        } else {
            if (r < max_batch) mp[r] = r * k + j;
        }
    }
}

void launch_init_maps(hipStream_t s, Engine& e) {
    int n = 2 * e.cfg.max_batch;
    k_init_maps<<<(n + 255) / 256, 256, 0, s>>>(e.ws.lm_map_d, e.ws.ident_map, e.cfg.max_batch, e.cfg.k);
}

// ===========================================================================
// Row planning + embedding gather (+ steering injection for drafter rows).
// One block per row.  Inactive rows get position -1 and a zero residual.
// ===========================================================================
struct PlanArgs {
    int kind, j, k, batch, cap, vocab, d, chunk, max_prompt;
    const int32_t *t, *len_d, *done, *hist, *drafts, *prompt_tok, *prompt_len;
    const float* steer;
    int add_steer;
    const float* row_add;  // [rows][d] added to every active row's embedding, or null
    int32_t *row_pos, *row_seq;
    float* x;
    float* ss;   // [rows][d/16]
    const void* embed;
};

template <typename TW>
__global__ __launch_bounds__(256) void k_plan_embed(PlanArgs a) {
    int r = blockIdx.x;
    int b, pos = -1, tok = 0;
    bool active = false;
    if (a.kind == kPlanDraft1) {
        b = r >> 1;
        int i = r & 1;
        if (b < a.batch && !a.done[b]) {
            int t = a.t[b], m = t - a.len_d[b];
            if (i == 1) { pos = t - 1; active = true; }
            else if (m == 2) { pos = t - 2; active = true; }
            if (active) tok = a.hist[(size_t)b * a.cap + pos];
        }
    } else if (a.kind == kPlanDraftJ) {
        b = r;
        if (b < a.batch && !a.done[b]) {
            pos = a.t[b] + a.j - 2;
            tok = a.drafts[b * a.k + a.j - 2];
            active = true;
        }
    } else if (a.kind == kPlanVerify) {
        b = r / (a.k + 1);
        int i = r % (a.k + 1);
        if (b < a.batch && !a.done[b]) {
            int t = a.t[b];
            pos = t - 1 + i;
            tok = i == 0 ? a.hist[(size_t)b * a.cap + t - 1] : a.drafts[b * a.k + i - 1];
            active = true;
        }
    } else {  // prefill chunk
        b = r / a.chunk;
        int i = r % a.chunk;
        pos = a.j * a.chunk + i;
        if (b < a.batch && pos < min(a.prompt_len[b], a.max_prompt) - 1) {
            tok = a.prompt_tok[(size_t)b * a.max_prompt + pos];
            active = true;
        }
    }
    if (!active) pos = -1;
    tok = tok < 0 ? 0 : (tok >= a.vocab ? a.vocab - 1 : tok);
    if (threadIdx.x == 0) {
        a.row_pos[r] = pos;
        a.row_seq[r] = b;
    }
    float* xr = a.x + (size_t)r * a.d;
    const TW* er = (const TW*)a.embed + (size_t)tok * a.d;
    const float* sr = a.steer + (size_t)b * a.d;
    const int nsl = a.d / 16;
    for (int sl = threadIdx.x; sl < nsl; sl += blockDim.x) {
        float acc = 0.0f;
        for (int c = 0; c < 16; ++c) {
            int i = sl * 16 + c;
            float v = 0.0f;
            if (active) {
                v = load_scalar<TW>(er, i);
                if (a.add_steer) v += sr[i];
                if (a.row_add) v += a.row_add[(size_t)r * a.d + i];
            }
            xr[i] = v;
            acc += v * v;
        }
        a.ss[(size_t)r * nsl + sl] = acc;
    }
}

void launch_plan_embed(hipStream_t s, Engine& e, ModelDev& m, int kind, int j, int rows, const int32_t* prompt_tok,
                       const int32_t* prompt_len, int max_prompt, int chunk, const float* row_add) {
    PlanArgs a;
    a.row_add = row_add;
    a.kind = kind; a.j = j; a.k = e.cfg.k; a.batch = e.batch; a.cap = e.cap; a.vocab = m.dm.vocab;
    a.d = m.dm.d_model; a.chunk = chunk; a.max_prompt = max_prompt;
    a.t = e.ws.t; a.len_d = e.ws.len_d; a.done = e.ws.done; a.hist = e.ws.hist; a.drafts = e.ws.drafts;
    a.prompt_tok = prompt_tok; a.prompt_len = prompt_len;
    a.steer = e.ws.steer;
    a.add_steer = !e.mlp && e.w_steer && (&m == &e.md) && (kind == kPlanDraft1 || kind == kPlanDraftJ);
    a.row_pos = e.ws.row_pos; a.row_seq = e.ws.row_seq; a.x = m.x; a.ss = m.ss; a.embed = m.embed;
    prof_begin(&e, kProfOther, 0.0);
    if (e.bf16) k_plan_embed<uint16_t><<<rows, 256, 0, s>>>(a);
    else k_plan_embed<float><<<rows, 256, 0, s>>>(a);
    prof_end(&e);
}

// ===========================================================================
// GEMV: Y[m][n] (op)= sum_k W[n][k] * Xn[m][k], Xn = optional RMSNorm(X) * gamma.
// W is streamed once per M-tile of rows; X rows are staged in LDS as fp32.
// Segments let one launch cover Q|K|V (concatenated output columns) or gate|up
// (paired rows, SwiGLU epilogue silu(gate) * up).
// ===========================================================================
struct GemvArgs {
    const float* X;
    const int32_t* in_map;
    int M, K;
    const void* gamma;
    float eps;
    const void* W[3];
    int seg_rows[3];
    int seg_off[3];
    int nseg, N, epi;
    float* Y;
    int ldy;
    const int32_t* out_map;
    const float* ubias;       // MLP steering: bias rows per sequence (row_seq), added to up (SwiGLU) or
                              // to the output (Add), or null
    int ub_ld;
    const int32_t* row_seq;
};

constexpr int kGemvThreads = 256;
constexpr int kGemvRowsPerWave = 4;
constexpr int kGemvRowsPerBlock = kGemvRowsPerWave * (kGemvThreads / kWave);

template <typename TW>
struct Vec16;
template <>
struct Vec16<uint16_t> {
    static constexpr int N = 8;
    __device__ static void load(const uint16_t* p, float* w) {
        uint4 u = *(const uint4*)p;
        w[0] = bf16_lo(u.x); w[1] = bf16_hi(u.x); w[2] = bf16_lo(u.y); w[3] = bf16_hi(u.y);
        w[4] = bf16_lo(u.z); w[5] = bf16_hi(u.z); w[6] = bf16_lo(u.w); w[7] = bf16_hi(u.w);
    }
};
template <>
struct Vec16<float> {
    static constexpr int N = 4;
    __device__ static void load(const float* p, float* w) {
        float4 u = *(const float4*)p;
        w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
    }
};

template <typename TW, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_gemv_vec(GemvArgs a) {
    extern __shared__ float xs[];  // [MT][K]
    __shared__ float red[kGemvThreads / kWave];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int K = a.K;
    const int m0 = blockIdx.y * MT;
    const int mc = min(MT, a.M - m0);

    // ---- prologue: gather, optionally RMS-normalise, stage in LDS ----
    for (int m = 0; m < MT; ++m) {
        float* xr = xs + (size_t)m * K;
        int src = -1;
        if (m < mc) src = a.in_map ? a.in_map[m0 + m] : m0 + m;
        float ss = 0.0f;
        for (int k = tid; k < K; k += kGemvThreads) {
            float v = src >= 0 ? a.X[(size_t)src * K + k] : 0.0f;
            xr[k] = v;
            ss += v * v;
        }
        if (a.gamma) {
            ss = wave_sum(ss);
            if (lane == 0) red[wave] = ss;
            __syncthreads();
            float tot = 0.0f;
            for (int w = 0; w < kGemvThreads / kWave; ++w) tot += red[w];
            float sc = rsqrtf(tot / (float)K + a.eps);
            for (int k = tid; k < K; k += kGemvThreads) xr[k] = xr[k] * sc * load_scalar<TW>((const TW*)a.gamma, k);
            __syncthreads();
        }
    }
    __syncthreads();

    constexpr int VN = Vec16<TW>::N;
    for (int rr = 0; rr < kGemvRowsPerWave; ++rr) {
        const int n = blockIdx.x * kGemvRowsPerBlock + wave * kGemvRowsPerWave + rr;
        if (n >= a.N) break;
        float acc0[MT], acc1[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) { acc0[m] = 0.0f; acc1[m] = 0.0f; }
        const TW* wr0;
        const TW* wr1 = nullptr;
        if (a.epi == kEpiSwiglu) {
            wr0 = (const TW*)a.W[0] + (size_t)n * K;
            wr1 = (const TW*)a.W[1] + (size_t)n * K;
        } else {
            int sgi = 0;
            while (sgi + 1 < a.nseg && n >= a.seg_off[sgi + 1]) ++sgi;
            wr0 = (const TW*)a.W[sgi] + (size_t)(n - a.seg_off[sgi]) * K;
        }
        for (int k = lane * VN; k < K; k += kWave * VN) {
            float w[VN];
            Vec16<TW>::load(wr0 + k, w);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const float* xv = xs + (size_t)m * K + k;
                float sacc = 0.0f;
#pragma unroll
                for (int e2 = 0; e2 < VN; ++e2) sacc += w[e2] * xv[e2];
                acc0[m] += sacc;
            }
            if (wr1) {
                Vec16<TW>::load(wr1 + k, w);
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const float* xv = xs + (size_t)m * K + k;
                    float sacc = 0.0f;
#pragma unroll
                    for (int e2 = 0; e2 < VN; ++e2) sacc += w[e2] * xv[e2];
                    acc1[m] += sacc;
                }
            }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            acc0[m] = wave_sum(acc0[m]);
            if (wr1) acc1[m] = wave_sum(acc1[m]);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (lane == m && m < mc) {
                int orow = a.out_map ? a.out_map[m0 + m] : m0 + m;
                if (orow >= 0) {
                    float* yp = a.Y + (size_t)orow * a.ldy + n;
                    if (a.epi == kEpiStore) {
                        *yp = acc0[m];
                    } else if (a.epi == kEpiAdd) {
                        float add = acc0[m];
                        if (a.ubias) add += a.ubias[(size_t)a.row_seq[m0 + m] * a.ub_ld + n];
                        *yp += add;
                    } else {
                        float up = acc1[m];
                        if (a.ubias) up += a.ubias[(size_t)a.row_seq[m0 + m] * a.ub_ld + n];
                        *yp = silu(acc0[m]) * up;
                    }
                }
            }
        }
    }
}

void launch_gemv(Engine* e, hipStream_t s, bool bf16, const float* X, const int32_t* in_map, int M, int K,
                 const void* gamma, float eps, const void* const* W, const int* seg_rows, int nseg, int epi, float* Y,
                 int ldy, const int32_t* out_map, const float* ubias, int ub_ld, const int32_t* row_seq) {
    GemvArgs a;
    a.ubias = ubias; a.ub_ld = ub_ld; a.row_seq = row_seq;
    a.X = X; a.in_map = in_map; a.M = M; a.K = K; a.gamma = gamma; a.eps = eps;
    int off = 0;
    for (int i = 0; i < 3; ++i) {
        a.W[i] = i < nseg ? W[i] : nullptr;
        a.seg_rows[i] = i < nseg ? seg_rows[i] : 0;
        a.seg_off[i] = off;
        off += a.seg_rows[i];
    }
    a.nseg = nseg;
    a.N = epi == kEpiSwiglu ? seg_rows[0] : off;
    a.epi = epi; a.Y = Y; a.ldy = ldy; a.out_map = out_map;
    // rows staged per pass: as many as fit 64 KiB of LDS, at most 8
    int mt = 8;
    while (mt > 1 && (mt / 2 >= M || (size_t)mt * K * 4 > 65536)) mt >>= 1;
    dim3 grid((a.N + kGemvRowsPerBlock - 1) / kGemvRowsPerBlock, (M + mt - 1) / mt);
    size_t sh = (size_t)mt * K * 4;
    // algorithmic bytes: every weight once, the input rows once, the output rows once
    double wrows = (double)(epi == kEpiSwiglu ? 2 * a.N : a.N);
    double nout = (double)a.N;
    prof_begin(e, kProfGemv, wrows * K * (bf16 ? 2.0 : 4.0) + (double)M * K * 4.0 + (double)M * nout * 4.0);
#define SD2_GEMV_CASE(MTV)                                                                  \
    case MTV:                                                                               \
        if (bf16) k_gemv_vec<uint16_t, MTV><<<grid, kGemvThreads, sh, s>>>(a);             \
        else k_gemv_vec<float, MTV><<<grid, kGemvThreads, sh, s>>>(a);                     \
        break;
    switch (mt) {
        SD2_GEMV_CASE(1)
        SD2_GEMV_CASE(2)
        SD2_GEMV_CASE(4)
        SD2_GEMV_CASE(8)
    }
#undef SD2_GEMV_CASE
    prof_end(e);
}

// ===========================================================================
// RoPE (rotate-half) on q in place and on k; append k, v of every active row to the cache.
// ===========================================================================
struct RopeArgs {
    float* qkv;
    int qkv_dim, H, Hkv, hd, cap, max_batch, layer;
    const int32_t *row_pos, *row_seq;
    const float *cosv, *sinv;
    float *kc, *vc;
};

__global__ __launch_bounds__(128) void k_rope_append(RopeArgs a) {
    int r = blockIdx.x;
    int pos = a.row_pos[r];
    if (pos < 0) return;
    int b = a.row_seq[r];
    int half = a.hd / 2;
    float* q = a.qkv + (size_t)r * a.qkv_dim;
    float* k = q + a.H * a.hd;
    const float* v = k + a.Hkv * a.hd;
    const float* cr = a.cosv + (size_t)pos * half;
    const float* sr = a.sinv + (size_t)pos * half;
    for (int idx = threadIdx.x; idx < a.H * half; idx += blockDim.x) {
        int h = idx / half, i = idx % half;
        float* qh = q + h * a.hd;
        float x0 = qh[i], x1 = qh[i + half], c = cr[i], sn = sr[i];
        qh[i] = x0 * c - x1 * sn;
        qh[i + half] = x1 * c + x0 * sn;
    }
    size_t base = ((size_t)a.layer * a.max_batch + b) * a.Hkv;
    for (int idx = threadIdx.x; idx < a.Hkv * half; idx += blockDim.x) {
        int h = idx / half, i = idx % half;
        const float* kh = k + h * a.hd;
        float x0 = kh[i], x1 = kh[i + half], c = cr[i], sn = sr[i];
        float* dst = a.kc + ((base + h) * a.cap + pos) * a.hd;
        dst[i] = x0 * c - x1 * sn;
        dst[i + half] = x1 * c + x0 * sn;
    }
    for (int idx = threadIdx.x; idx < a.Hkv * a.hd; idx += blockDim.x) {
        int h = idx / a.hd, i = idx % a.hd;
        a.vc[((base + h) * a.cap + pos) * a.hd + i] = v[idx];
    }
}

// ===========================================================================
// One decoder layer on `rows` planned rows.
// ===========================================================================
static WsCall ws_base(Engine& e, ModelDev& m) {
    WsCall c{};
    c.part = e.ws.ws_part;
    c.cnt = e.ws.ws_cnt;
    c.eps = m.dm.rms_eps;
    c.nss = m.dm.d_model / 16;
    return c;
}

void launch_layer(hipStream_t s, Engine& e, ModelDev& m, int layer, int rows, int rps, const float* ubias,
                  int ub_ld, bool bias_after, const int32_t* ub_map) {
    const int32_t* bias_rows = ub_map ? ub_map : e.ws.row_seq;
    const float* up_bias = bias_after ? nullptr : ubias;
    const float* out_bias = bias_after ? ubias : nullptr;
    const sd2_dims& dm = m.dm;
    const void* const* W = m.layer + (size_t)layer * 9;
    int hd = m.hd, H = dm.n_heads, Hkv = dm.n_kv_heads;
    if (e.bf16) {
        // Q|K|V with the attention RMSNorm as prologue, RoPE and the cache append as epilogue
        WsCall c = ws_base(e, m);
        c.X = m.x; c.M = rows; c.K = dm.d_model; c.gamma = W[kAttnNorm]; c.ss = m.ss;
        c.W[0] = W[kWq]; c.W[1] = W[kWk]; c.W[2] = W[kWv];
        c.seg_rows[0] = H * hd; c.seg_rows[1] = Hkv * hd; c.seg_rows[2] = Hkv * hd;
        c.nseg = 3; c.mode = kEpiQkv;
        c.H = H; c.Hkv = Hkv; c.hd = hd; c.row_pos = e.ws.row_pos; c.row_seq = e.ws.row_seq;
        c.rcos = m.rope_cos; c.rsin = m.rope_sin; c.qout = e.ws.qkv; c.kc = m.kc; c.vc = m.vc;
        c.cap = e.cap; c.max_batch = e.cfg.max_batch; c.layer = layer;
        launch_wsgemv(&e, s, c);
        launch_attn(e, s, m, layer, rows, rps, e.ws.qkv, H * hd);
        // O projection + residual (+ slice sums of squares for the FFN norm)
        WsCall o = ws_base(e, m);
        o.X = e.ws.attn; o.M = rows; o.K = H * hd; o.W[0] = W[kWo]; o.seg_rows[0] = dm.d_model; o.nseg = 1;
        o.mode = kEpiAdd; o.Y = m.x; o.ldy = dm.d_model; o.ss_out = m.ss;
        launch_wsgemv(&e, s, o);
        // gate|up with the FFN RMSNorm prologue and SwiGLU epilogue
        WsCall g = ws_base(e, m);
        g.X = m.x; g.M = rows; g.K = dm.d_model; g.gamma = W[kFfnNorm]; g.ss = m.ss;
        g.W[0] = W[kWg]; g.W[1] = W[kWu]; g.seg_rows[0] = dm.d_ff; g.seg_rows[1] = dm.d_ff; g.nseg = 2;
        g.mode = kEpiSwiglu; g.Y = e.ws.ffh; g.ldy = dm.d_ff;
        g.ubias = up_bias; g.ub_ld = ub_ld; g.row_seq = bias_rows;
        launch_wsgemv(&e, s, g);
        // down projection + residual
        WsCall d = ws_base(e, m);
        d.X = e.ws.ffh; d.M = rows; d.K = dm.d_ff; d.W[0] = W[kWd]; d.seg_rows[0] = dm.d_model; d.nseg = 1;
        d.mode = kEpiAdd; d.Y = m.x; d.ldy = dm.d_model; d.ss_out = m.ss;
        d.ubias = out_bias; d.ub_ld = ub_ld; d.row_seq = bias_rows;
        launch_wsgemv(&e, s, d);
        return;
    }
    // fp32 weights: vector projections, separate RoPE/append
    {
        const void* ws[3] = {W[kWq], W[kWk], W[kWv]};
        int rws[3] = {H * hd, Hkv * hd, Hkv * hd};
        launch_gemv(&e, s, e.bf16, m.x, nullptr, rows, dm.d_model, W[kAttnNorm], dm.rms_eps, ws, rws, 3, kEpiStore,
                    e.ws.qkv, m.qkv_dim, nullptr);
    }
    {
        RopeArgs a;
        a.qkv = e.ws.qkv; a.qkv_dim = m.qkv_dim; a.H = H; a.Hkv = Hkv; a.hd = hd; a.cap = e.cap;
        a.max_batch = e.cfg.max_batch; a.layer = layer; a.row_pos = e.ws.row_pos; a.row_seq = e.ws.row_seq;
        a.cosv = m.rope_cos; a.sinv = m.rope_sin; a.kc = m.kc; a.vc = m.vc;
        prof_begin(&e, kProfOther, 0.0);
        k_rope_append<<<rows, 128, 0, s>>>(a);
        prof_end(&e);
    }
    launch_attn(e, s, m, layer, rows, rps, e.ws.qkv, m.qkv_dim);
    {
        const void* ws[1] = {W[kWo]};
        int rws[1] = {dm.d_model};
        launch_gemv(&e, s, e.bf16, e.ws.attn, nullptr, rows, H * hd, nullptr, 0.f, ws, rws, 1, kEpiAdd, m.x,
                    dm.d_model, nullptr);
    }
    {
        const void* ws[2] = {W[kWg], W[kWu]};
        int rws[2] = {dm.d_ff, dm.d_ff};
        launch_gemv(&e, s, e.bf16, m.x, nullptr, rows, dm.d_model, W[kFfnNorm], dm.rms_eps, ws, rws, 2, kEpiSwiglu,
                    e.ws.ffh, dm.d_ff, nullptr, up_bias, ub_ld, bias_rows);
    }
    {
        const void* ws[1] = {W[kWd]};
        int rws[1] = {dm.d_model};
        launch_gemv(&e, s, e.bf16, e.ws.ffh, nullptr, rows, dm.d_ff, nullptr, 0.f, ws, rws, 1, kEpiAdd, m.x,
                    dm.d_model, nullptr, out_bias, ub_ld, bias_rows);
    }
}

void launch_lm_head(Engine& e, ModelDev& m, int rows, float* Y, const int32_t* out_map) {
    if (e.bf16) {
        WsCall c = ws_base(e, m);
        c.X = m.x; c.M = rows; c.K = m.dm.d_model; c.gamma = m.final_norm; c.ss = m.ss;
        c.W[0] = m.lm_head; c.seg_rows[0] = m.dm.vocab; c.nseg = 1; c.mode = kEpiStore;
        c.Y = Y; c.ldy = m.dm.vocab; c.out_map = out_map;
        launch_wsgemv(&e, e.stream, c);
        return;
    }
    const void* ws[1] = {m.lm_head};
    int rws[1] = {m.dm.vocab};
    launch_gemv(&e, e.stream, e.bf16, m.x, nullptr, rows, m.dm.d_model, m.final_norm, m.dm.rms_eps, ws, rws, 1,
                kEpiStore, Y, m.dm.vocab, out_map);
}

void launch_steer(Engine& e, const float* X, const float* ss, const int32_t* in_map, int rows) {
    if (e.bf16) {
        WsCall c = ws_base(e, e.mv);
        c.X = X; c.in_map = in_map; c.M = rows; c.K = e.mv.dm.d_model; c.gamma = e.mv.final_norm; c.ss = ss;
        c.W[0] = e.w_steer; c.seg_rows[0] = e.md.dm.d_model; c.nseg = 1; c.mode = kEpiStore;
        c.Y = e.ws.steer; c.ldy = e.md.dm.d_model;
        launch_wsgemv(&e, e.stream, c);
        return;
    }
    const void* ws[1] = {e.w_steer};
    int rws[1] = {e.md.dm.d_model};
    launch_gemv(&e, e.stream, e.bf16, X, in_map, rows, e.mv.dm.d_model, e.mv.final_norm, e.mv.dm.rms_eps, ws, rws,
                1, kEpiStore, e.ws.steer, e.md.dm.d_model, nullptr);
}

// ===========================================================================
// MLP steering (eq. (2)): taps of the verifier's residual stream, g = LayerNorm(W_hml [h; m; l]),
// per-layer up-projection biases W_s g.
// ===========================================================================
// Residual rows after `layer` into every tap slot taken there (per-operation verify pass).
__global__ void k_tap_copy(const float* x, int d, int rows, int maxm, float* taps, int m0, int m1, int m2) {
    const int r = blockIdx.x;
    const int mask = m0 | (m1 << 1) | (m2 << 2);
    for (int sl = 0; sl < 3; ++sl) {
        if (!((mask >> sl) & 1)) continue;
        float* dst = taps + ((size_t)sl * maxm + r) * d;
        for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = x[(size_t)r * d + i];
    }
}

void launch_tap_copy(hipStream_t s, Engine& e, int layer, int rows) {
    const int* tl = e.tap_layer;
    if (tl[0] != layer && tl[1] != layer && tl[2] != layer) return;
    prof_begin(&e, kProfOther, 0.0);
    k_tap_copy<<<rows, 256, 0, s>>>(e.mv.x, e.mv.dm.d_model, rows, e.maxm, e.ws.taps, tl[0] == layer,
                                    tl[1] == layer, tl[2] == layer);
    prof_end(&e);
}

// Prefill: the tap rows at position len-2 of each sequence go straight to its [h; m; l] row.
__global__ void k_prefill_tap(const int32_t* row_pos, const int32_t* row_seq, const int32_t* prompt_len,
                              int max_prompt, const float* x, int d, float* tapsel, int batch, int m0, int m1,
                              int m2) {
    const int r = blockIdx.x;
    const int pos = row_pos[r];
    if (pos < 0) return;
    const int b = row_seq[r];
    if (b >= batch || pos != min(prompt_len[b], max_prompt) - 2) return;
    const int mask = m0 | (m1 << 1) | (m2 << 2);
    for (int sl = 0; sl < 3; ++sl) {
        if (!((mask >> sl) & 1)) continue;
        float* dst = tapsel + ((size_t)b * 3 + sl) * d;
        for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = x[(size_t)r * d + i];
    }
}

void launch_prefill_tap(hipStream_t s, Engine& e, int layer, int rows, const int32_t* prompt_len, int max_prompt) {
    const int* tl = e.tap_layer;
    if (tl[0] != layer && tl[1] != layer && tl[2] != layer) return;
    k_prefill_tap<<<rows, 256, 0, s>>>(e.ws.row_pos, e.ws.row_seq, prompt_len, max_prompt, e.mv.x,
                                       e.mv.dm.d_model, e.ws.tapsel, e.batch, tl[0] == layer, tl[1] == layer,
                                       tl[2] == layer);
}

// [h; m; l] of row in_map[b] (identity when null) of three [rows][d] sources.
__global__ void k_tap_gather(const float* s0, const float* s1, const float* s2, const int32_t* in_map, int d,
                             float* tapsel) {
    const int b = blockIdx.x;
    const int r = in_map ? in_map[b] : b;
    const float* src[3] = {s0, s1, s2};
    for (int sl = 0; sl < 3; ++sl)
        for (int i = threadIdx.x; i < d; i += blockDim.x)
            tapsel[((size_t)b * 3 + sl) * d + i] = src[sl][(size_t)r * d + i];
}

// In-place LayerNorm of rows [rows][d]: (g - mean) / sqrt(var + eps) * gain + shift, population
// variance; one workgroup per row, two passes over it (mean, then centred squares).
template <typename TW>
__global__ __launch_bounds__(256) void k_layernorm_rows(float* X, int d, const TW* gain, const TW* shift, float eps) {
    __shared__ float red[4];
    __shared__ float stat[2];
    float* x = X + (size_t)blockIdx.x * d;
    const int lane = threadIdx.x & 63, wave = threadIdx.x / 64;
    float sum = 0.0f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) sum += x[i];
    sum = wave_sum(sum);
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) stat[0] = (red[0] + red[1] + red[2] + red[3]) / (float)d;
    __syncthreads();
    const float mean = stat[0];
    float sq = 0.0f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
        const float c = x[i] - mean;
        sq += c * c;
    }
    sq = wave_sum(sq);
    if (lane == 0) red[wave] = sq;
    __syncthreads();
    if (threadIdx.x == 0) stat[1] = rsqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
    __syncthreads();
    const float inv = stat[1];
    for (int i = threadIdx.x; i < d; i += blockDim.x)
        x[i] = (x[i] - mean) * inv * load_scalar<TW>(gain, i) + load_scalar<TW>(shift, i);
}

// Y[rows][N] = X[rows][K] . W^T: the MFMA projection kernel when it has a plan for the shape,
// else the vector kernel (small K, or f32 weights).
static void project_rows(Engine& e, const float* X, int rows, int K, const void* W, int N, float* Y) {
    if (e.bf16 && ws_plan(rows < 16 ? rows : 16, N, K, kEpiStore).S) {
        WsCall c = ws_base(e, e.mv);
        c.X = X; c.M = rows; c.K = K;
        c.W[0] = W; c.seg_rows[0] = N; c.nseg = 1; c.mode = kEpiStore;
        c.Y = Y; c.ldy = N;
        launch_wsgemv(&e, e.stream, c);
        return;
    }
    const void* ws[1] = {W};
    int rws[1] = {N};
    launch_gemv(&e, e.stream, e.bf16, X, nullptr, rows, K, nullptr, 0.f, ws, rws, 1, kEpiStore, Y, N, nullptr);
}

void launch_mlp_steer(Engine& e, const float* const* src, const int32_t* in_map, int rows) {
    const int dV = e.mv.dm.d_model;
    const int nb = e.nbias;
    if (src) {  // else tapsel already holds the rows (prefill)
        prof_begin(&e, kProfOther, 0.0);
        k_tap_gather<<<rows, 256, 0, e.stream>>>(src[0], src[1], src[2], in_map, dV, e.ws.tapsel);
        prof_end(&e);
    }
    project_rows(e, e.ws.tapsel, rows, 3 * dV, e.w_hml, dV, e.ws.gsteer);
    prof_begin(&e, kProfOther, 0.0);
    if (e.bf16)
        k_layernorm_rows<uint16_t><<<rows, 256, 0, e.stream>>>(e.ws.gsteer, dV, (const uint16_t*)e.ln_gain,
                                                               (const uint16_t*)e.ln_bias, e.ln_eps);
    else
        k_layernorm_rows<float><<<rows, 256, 0, e.stream>>>(e.ws.gsteer, dV, (const float*)e.ln_gain,
                                                            (const float*)e.ln_bias, e.ln_eps);
    prof_end(&e);
    project_rows(e, e.ws.gsteer, rows, dV, e.w_steer, nb, e.ws.ubias);
}

// Conditional bias, hidden layer: h = SiLU(h + c_l of the row's sequence), in place, [rows][R].
__global__ void k_cond_act(float* h, int R, const float* c, int c_ld, const int32_t* row_seq) {
    const int r = blockIdx.x;
    const float* cr = c + (size_t)row_seq[r] * c_ld;
    for (int i = threadIdx.x; i < R; i += blockDim.x) h[(size_t)r * R + i] = silu(h[(size_t)r * R + i] + cr[i]);
}

void launch_cond_bias(hipStream_t s, Engine& e, int layer, int rows) {
    const int R = e.cfg.cond_rank, d = e.md.dm.d_model, F = e.md.dm.d_ff;
    const size_t es = e.bf16 ? 2 : 4;
    // V_l^f f: the raw residual rows as they enter the layer (no norm)
    project_rows(e, e.md.x, rows, d, (const char*)e.w_cf + (size_t)layer * R * d * es, R, e.ws.cond_h);
    prof_begin(&e, kProfOther, 0.0);
    k_cond_act<<<rows, 256, 0, s>>>(e.ws.cond_h, R, e.ws.ubias + (size_t)layer * R, e.nbias, e.ws.row_seq);
    prof_end(&e);
    project_rows(e, e.ws.cond_h, rows, R, (const char*)e.w_cu + (size_t)layer * F * R * es, F, e.ws.cond_b);
}

// ===========================================================================
// Sampler.  Vocabulary rows are cut into kVocabChunks slices; each slice writes a
// partial, and one wave per sequence combines the 64 partials in a fixed order.
// ===========================================================================
struct SampArgs {
    const float *logits_v, *logits_d;
    int V, k, batch, chunk;  // chunk: slice length, a multiple of 4
    float T;
    uint64_t seed;
    const int32_t *t, *done;
    int32_t *drafts, *own_drafts, *n_eff, *own_n, *own_y, *steer_map;
    const int32_t *forced, *forced_on;
    VPart* part;
    float *lse_v, *lse_d;
    int32_t* argmax_v;
    int32_t* nonfinite;  // set to 1 when a logit read here is a NaN or an infinity
    int j;
    int32_t *out_tokens, *out_counts, *len_v, *len_d, *produced, *hist, *tt, *done_w;
    int cap, max_new;
};

__device__ __forceinline__ int clamp_tok(int v, int V) { return v < 0 ? 0 : (v >= V ? V - 1 : v); }

__device__ __forceinline__ void store_through_i(int32_t* p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void block_argbest(ArgBest& a, ArgBest* sh) {
    int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    a = wave_argbest(a);
    __syncthreads();
    if (lane == 0) sh[wave] = a;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < (int)(blockDim.x / kWave); ++w)
            if (better(sh[w].s, sh[w].i, a.s, a.i)) a = sh[w];
    }
}

// Draft pick, partial: best of l/T + Gumbel (or l when greedy) over one vocabulary slice.
__global__ __launch_bounds__(256) void k_pick_partial(SampArgs a) {
    __shared__ ArgBest sh[4];
    int c = blockIdx.x, b = blockIdx.y;
    const float* row = a.logits_d + ((size_t)b * a.k + (a.j - 1)) * a.V;
    int v0 = c * a.chunk, v1 = min(a.V, v0 + a.chunk);
    uint32_t t = (uint32_t)a.t[b];
    ArgBest best{-INFINITY, 0x7fffffff};
    for (int q = v0 + 4 * threadIdx.x; q < v1; q += 4 * blockDim.x) {
        // the 4 logits are read unconditionally (index clamped) before any comparison, so the
        // loads are not serialised behind per-element branches
        float r4[4];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) r4[e2] = row[min(q + e2, v1 - 1)];
        if (a.T > 0.0f) {
            U4 w = philox10(U4{(uint32_t)q >> 2, (uint32_t)a.j, t, (kDraft << 24) | (uint32_t)b}, (uint32_t)a.seed,
                            (uint32_t)(a.seed >> 32));
            uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                if (q + e2 >= v1) break;
                float sc = r4[e2] / a.T + gumbel(ws[e2]);
                if (better(sc, q + e2, best.s, best.i)) best = ArgBest{sc, q + e2};
            }
        } else {
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                if (q + e2 >= v1) break;
                float sc = r4[e2];
                if (better(sc, q + e2, best.s, best.i)) best = ArgBest{sc, q + e2};
            }
        }
    }
    block_argbest(best, sh);
    if (threadIdx.x == 0) {
        VPart& p = a.part[(size_t)b * kVocabChunks + c];
        p.best = best.s;
        p.idx = best.i;
    }
}

// Draft pick, final: combine the slices; record the library's own draft and the effective one.
__global__ __launch_bounds__(64) void k_pick_final(SampArgs a) {
    int b = blockIdx.x, lane = threadIdx.x;
    const VPart& p = a.part[(size_t)b * kVocabChunks + lane];
    ArgBest best = wave_argbest(ArgBest{p.best, p.idx});
    if (lane == 0) {
        int own = best.i;
        int eff = *a.forced_on ? clamp_tok(a.forced[b * (a.k + 2) + a.j - 1], a.V) : own;
        a.own_drafts[b * a.k + a.j - 1] = own;
        a.drafts[b * a.k + a.j - 1] = eff;
    }
}

void launch_draft_pick(hipStream_t s, Engine& e, int j);

// Log-normaliser partials of the 2k+1 rows of each sequence (k+1 verifier rows, then k
// drafter rows); greedy mode computes argmax partials of the verifier rows instead.
__global__ __launch_bounds__(256) void k_row_partial(SampArgs a) {
    __shared__ float shm[4], shs[4];
    __shared__ ArgBest sha[4];
    int c = blockIdx.x, rowid = blockIdx.y;
    int per = 2 * a.k + 1;
    int b = rowid / per, i = rowid % per;
    const float* row = i <= a.k ? a.logits_v + ((size_t)b * (a.k + 1) + i) * a.V
                                : a.logits_d + ((size_t)b * a.k + (i - a.k - 1)) * a.V;
    int v0 = c * a.chunk, v1 = min(a.V, v0 + a.chunk);
    VPart& p = a.part[(size_t)rowid * kVocabChunks + c];
    // every logit of the round's 2k+1 rows passes here: any NaN or infinity raises the flag
    bool nonfinite = false;
    if (a.T > 0.0f) {
        float m = -INFINITY, sm = 0.0f;
        // 8 logits per thread are read (index clamped) before they are merged, in the same order
        for (int vb = v0 + threadIdx.x; vb < v1; vb += 8 * blockDim.x) {
            float x[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) x[i] = row[min(vb + i * (int)blockDim.x, v1 - 1)];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                nonfinite |= !isfinite(x[i]);
                if (vb + i * (int)blockDim.x < v1) lse_merge(m, sm, x[i] / a.T, 1.0f);
            }
        }
        wave_lse(m, sm);
        int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
        if (lane == 0) { shm[wave] = m; shs[wave] = sm; }
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int w = 1; w < (int)(blockDim.x / kWave); ++w) lse_merge(m, sm, shm[w], shs[w]);
            p.m = m;
            p.s = sm;
        }
    } else {
        // greedy: argmax partials of the verifier rows; the drafter rows are only checked
        ArgBest best{-INFINITY, 0x7fffffff};
        for (int vb = v0 + threadIdx.x; vb < v1; vb += 8 * blockDim.x) {
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = row[min(vb + e * (int)blockDim.x, v1 - 1)];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                nonfinite |= !isfinite(x[e]);
                const int v = vb + e * (int)blockDim.x;
                if (i <= a.k && v < v1 && better(x[e], v, best.s, best.i)) best = ArgBest{x[e], v};
            }
        }
        block_argbest(best, sha);
        if (threadIdx.x == 0) { p.best = best.s; p.idx = best.i; }
    }
    // one store of 1 (idempotent: no read-modify-write needed) per workgroup that saw one
    if (__syncthreads_or(nonfinite) && threadIdx.x == 0) store_through_i(a.nonfinite, 1);
}

// Accept/reject: one wave per sequence.  Every row's partials and every draft's two logits are
// requested before any is used (lane i fetches draft i's pair), then lane 0 scans the drafts.
__global__ __launch_bounds__(64) void k_accept(SampArgs a) {
    int b = blockIdx.x, lane = threadIdx.x;
    int per = 2 * a.k + 1;
    __shared__ float lse[2 * kMaxK + 1];
    __shared__ int amax[kMaxK + 1];
    __shared__ float lpv[kMaxK], lqv[kMaxK];
    const int* dr = a.drafts + b * a.k;
    float xv = 0.f, xd = 0.f;
    if (a.T > 0.0f && lane < a.k) {
        const int x = dr[lane];
        xv = a.logits_v[((size_t)b * (a.k + 1) + lane) * a.V + x];
        xd = a.logits_d[((size_t)b * a.k + lane) * a.V + x];
    }
    // rows in batches of 8: the batch's loads (indices clamped, unconditional) and then its
    // independent wave reductions
    for (int i0 = 0; i0 < per; i0 += 8) {
        float f0[8], f1[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const VPart& p = a.part[((size_t)b * per + min(i0 + i, per - 1)) * kVocabChunks + lane];
            f0[i] = a.T > 0.0f ? p.m : p.best;
            f1[i] = a.T > 0.0f ? p.s : __int_as_float(p.idx);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = i0 + i;
            if (r >= per) break;
            if (a.T > 0.0f) {
                float m = f0[i], sm = f1[i];
                wave_lse(m, sm);
                if (lane == 0) lse[r] = m + logf(sm);
            } else if (r <= a.k) {
                ArgBest best = wave_argbest(ArgBest{f0[i], __float_as_int(f1[i])});
                if (lane == 0) amax[r] = best.i;
            }
        }
    }
    if (a.T > 0.0f && lane < a.k) {
        lpv[lane] = xv;
        lqv[lane] = xd;
    }
    __syncthreads();
    if (lane != 0) return;
    uint32_t t = (uint32_t)a.t[b];
    int n = 0;
    if (a.T > 0.0f) {
        for (int i = 0; i <= a.k; ++i) a.lse_v[b * (a.k + 1) + i] = lse[i];
        for (int i = 0; i < a.k; ++i) a.lse_d[b * a.k + i] = lse[a.k + 1 + i];
        for (int i = 0; i < a.k; ++i) {
            float lp = lpv[i] / a.T - lse[i];
            float lq = lqv[i] / a.T - lse[a.k + 1 + i];
            float ratio = lp - lq;
            float lu = logf(u01(rng_word(a.seed, (uint32_t)i, 0u, t, kAccept, (uint32_t)b, 0)));
            if (!(lu < ratio)) break;
            ++n;
        }
    } else {
        for (int i = 0; i <= a.k; ++i) a.argmax_v[b * (a.k + 1) + i] = amax[i];
        for (int i = 0; i < a.k; ++i) {
            if (dr[i] != amax[i]) break;
            ++n;
        }
    }
    int eff = *a.forced_on ? min(max(a.forced[b * (a.k + 2) + a.k], 0), a.k) : n;
    a.own_n[b] = n;
    a.n_eff[b] = eff;
    a.steer_map[b] = b * (a.k + 1) + eff;
    if (a.T == 0.0f) a.own_y[b] = amax[eff];
}

// Final draw, partial: residual (p - q)+ with Gumbel noise after a rejection, and the plain
// p-Gumbel score (bonus draw after full acceptance, or fallback for an empty residual).
__global__ __launch_bounds__(256) void k_final_partial(SampArgs a) {
    __shared__ ArgBest sh1[4], sh2[4];
    __shared__ int shf[4];
    int c = blockIdx.x, b = blockIdx.y;
    int n = a.n_eff[b];
    const float* pr = a.logits_v + ((size_t)b * (a.k + 1) + n) * a.V;
    const float* qr = n < a.k ? a.logits_d + ((size_t)b * a.k + n) * a.V : nullptr;
    float lp = a.lse_v[b * (a.k + 1) + n];
    float lq = n < a.k ? a.lse_d[b * a.k + n] : 0.0f;
    uint32_t t = (uint32_t)a.t[b];
    int v0 = c * a.chunk, v1 = min(a.V, v0 + a.chunk);
    ArgBest br{-INFINITY, 0x7fffffff}, bp{-INFINITY, 0x7fffffff};
    int flag = 0;
    for (int q = v0 + 4 * threadIdx.x; q < v1; q += 4 * blockDim.x) {
        U4 w = philox10(U4{(uint32_t)q >> 2, 0u, t, (kFinal << 24) | (uint32_t)b}, (uint32_t)a.seed,
                        (uint32_t)(a.seed >> 32));
        uint32_t ws[4] = {w.x, w.y, w.z, w.w};
        // the 4 logits of each row are read (index clamped) before any is used
        float p4[4], q4[4];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
            p4[e2] = pr[min(q + e2, v1 - 1)];
            q4[e2] = qr ? qr[min(q + e2, v1 - 1)] : 0.0f;
        }
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
            if (q + e2 >= v1) break;
            int v = q + e2;
            float g = gumbel(ws[e2]);
            float sp = p4[e2] / a.T + g;
            if (better(sp, v, bp.s, bp.i)) bp = ArgBest{sp, v};
            if (qr) {
                float p = expf(p4[e2] / a.T - lp);
                float qq = expf(q4[e2] / a.T - lq);
                float r = p - qq;
                if (r > 0.0f) {
                    flag = 1;
                    float sr = logf(r) + g;
                    if (better(sr, v, br.s, br.i)) br = ArgBest{sr, v};
                }
            }
        }
    }
    int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    int fl = __any(flag) ? 1 : 0;
    if (lane == 0) shf[wave] = fl;
    block_argbest(br, sh1);
    block_argbest(bp, sh2);
    if (threadIdx.x == 0) {
        int f = 0;
        for (int w = 0; w < (int)(blockDim.x / kWave); ++w) f |= shf[w];
        VPart& p = a.part[(size_t)b * kVocabChunks + c];
        p.best = br.s; p.idx = br.i; p.best2 = bp.s; p.idx2 = bp.i; p.flag = f;
    }
}

// Combine the final-draw slices, then commit: emit tokens, append history, roll back lengths.
__global__ __launch_bounds__(64) void k_commit(SampArgs a) {
    int b = blockIdx.x, lane = threadIdx.x;
    int y_own;
    if (a.T > 0.0f) {
        const VPart& p = a.part[(size_t)b * kVocabChunks + lane];
        int n = a.n_eff[b];
        bool res = (n < a.k) && __any(p.flag);
        ArgBest best = res ? wave_argbest(ArgBest{p.flag ? p.best : -INFINITY, p.flag ? p.idx : 0x7fffffff})
                           : wave_argbest(ArgBest{p.best2, p.idx2});
        y_own = best.i;
        if (lane == 0) a.own_y[b] = y_own;
    } else {
        y_own = a.own_y[b];
    }
    if (lane != 0) return;
    int y = *a.forced_on ? clamp_tok(a.forced[b * (a.k + 2) + a.k + 1], a.V) : y_own;
    int32_t* ot = a.out_tokens + b * (a.k + 1);
    if (b >= a.batch || a.done_w[b]) {
        a.out_counts[b] = 0;
        for (int i = 0; i <= a.k; ++i) ot[i] = -1;
        return;
    }
    int t = a.tt[b], n = a.n_eff[b];
    int remaining = a.max_new - a.produced[b];
    int count = min(n + 1, remaining);
    int32_t* hs = a.hist + (size_t)b * a.cap;
    for (int i = 0; i < n; ++i) hs[t + i] = a.drafts[b * a.k + i];
    hs[t + n] = y;
    for (int i = 0; i <= a.k; ++i) ot[i] = i < count ? hs[t + i] : -1;
    a.out_counts[b] = count;
    a.produced[b] += count;
    if (a.produced[b] >= a.max_new) a.done_w[b] = 1;
    a.len_v[b] = t + n;
    a.len_d[b] = min(t + a.k - 1, t + n);
    a.tt[b] = t + n + 1;
}

static SampArgs samp_args(Engine& e) {
    SampArgs a;
    a.logits_v = e.ws.logits_v; a.logits_d = e.ws.logits_d;
    a.V = e.mv.dm.vocab; a.k = e.cfg.k; a.batch = e.batch;
    a.chunk = ((a.V + kVocabChunks - 1) / kVocabChunks + 3) / 4 * 4;
    a.T = e.cfg.temperature; a.seed = e.cfg.seed;
    a.t = e.ws.t; a.done = e.ws.done;
    a.drafts = e.ws.drafts; a.own_drafts = e.ws.own_drafts; a.n_eff = e.ws.n_eff; a.own_n = e.ws.own_n;
    a.own_y = e.ws.own_y; a.steer_map = e.ws.steer_map;
    a.forced = e.ws.forced; a.forced_on = e.ws.forced_on;
    a.part = e.ws.part; a.lse_v = e.ws.lse_v; a.lse_d = e.ws.lse_d; a.argmax_v = e.ws.argmax_v;
    a.nonfinite = e.ws.nonfinite;
    a.j = 0;
    a.out_tokens = nullptr; a.out_counts = nullptr;
    a.len_v = e.ws.len_v; a.len_d = e.ws.len_d; a.produced = e.ws.produced; a.hist = e.ws.hist; a.tt = e.ws.t;
    a.done_w = e.ws.done;
    a.cap = e.cap; a.max_new = e.cfg.max_new_tokens;
    return a;
}

void launch_draft_pick(hipStream_t s, Engine& e, int j) {
    SampArgs a = samp_args(e);
    a.j = j;
    prof_begin(&e, kProfSampler, 0.0);
    k_pick_partial<<<dim3(kVocabChunks, e.batch), 256, 0, s>>>(a);
    k_pick_final<<<e.batch, 64, 0, s>>>(a);
    prof_end(&e);
}

void launch_verify_decide(hipStream_t s, Engine& e, int32_t* out_tokens, int32_t* out_counts) {
    SampArgs a = samp_args(e);
    a.out_tokens = out_tokens;
    a.out_counts = out_counts;
    int per = 2 * e.cfg.k + 1;
    prof_begin(&e, kProfSampler, 0.0);
    k_row_partial<<<dim3(kVocabChunks, e.batch * per), 256, 0, s>>>(a);
    k_accept<<<e.batch, 64, 0, s>>>(a);
    if (e.cfg.temperature > 0.0f) k_final_partial<<<dim3(kVocabChunks, e.batch), 256, 0, s>>>(a);
    k_commit<<<e.batch, 64, 0, s>>>(a);
    prof_end(&e);
}

// ===========================================================================
// Prefill helpers.
// ===========================================================================
// Keep the verifier residual of the row at position len-2 (the steering tap of the first round).
__global__ void k_prefill_capture(const int32_t* row_pos, const int32_t* row_seq, const int32_t* prompt_len,
                                  int max_prompt, const float* x, const float* ss, float* hcap, float* hcap_ss,
                                  int d, int batch) {
    int r = blockIdx.x;
    int pos = row_pos[r];
    if (pos < 0) return;
    int b = row_seq[r];
    if (b >= batch || pos != min(prompt_len[b], max_prompt) - 2) return;
    for (int i = threadIdx.x; i < d; i += blockDim.x) hcap[(size_t)b * d + i] = x[(size_t)r * d + i];
    for (int i = threadIdx.x; i < d / 16; i += blockDim.x) hcap_ss[(size_t)b * (d / 16) + i] = ss[(size_t)r * (d / 16) + i];
}

void launch_prefill_capture(hipStream_t s, Engine& e, int rows, const int32_t* prompt_len, int max_prompt) {
    k_prefill_capture<<<rows, 256, 0, s>>>(e.ws.row_pos, e.ws.row_seq, prompt_len, max_prompt, e.mv.x, e.mv.ss,
                                           e.ws.hcap, e.ws.hcap_ss, e.mv.dm.d_model, e.batch);
}

__global__ void k_prefill_finish(int batch, const int32_t* prompt_tok, const int32_t* prompt_len, int max_prompt,
                                 int32_t* hist, int cap, int32_t* t, int32_t* len_v, int32_t* len_d,
                                 int32_t* produced, int32_t* done, float* steer, int dD, int vocab, float* ubias,
                                 int nb) {
    int b = blockIdx.x;
    int p = min(max(prompt_len[b], 1), max_prompt);
    for (int i = threadIdx.x; i < p; i += blockDim.x) {
        int tok = prompt_tok[(size_t)b * max_prompt + i];
        hist[(size_t)b * cap + i] = tok < 0 ? 0 : (tok >= vocab ? vocab - 1 : tok);
    }
    if (p < 2) {
        for (int i = threadIdx.x; i < dD; i += blockDim.x) steer[(size_t)b * dD + i] = 0.0f;
        if (ubias)
            for (int i = threadIdx.x; i < nb; i += blockDim.x) ubias[(size_t)b * nb + i] = 0.0f;
    }
    if (threadIdx.x == 0) {
        t[b] = p;
        len_v[b] = p - 1;
        len_d[b] = p - 1;
        produced[b] = 0;
        done[b] = 0;
    }
}

void launch_prefill_finish(hipStream_t s, Engine& e, int batch, const int32_t* prompt_tok, const int32_t* prompt_len,
                           int max_prompt) {
    k_prefill_finish<<<batch, 256, 0, s>>>(batch, prompt_tok, prompt_len, max_prompt, e.ws.hist, e.cap, e.ws.t,
                                           e.ws.len_v, e.ws.len_d, e.ws.produced, e.ws.done, e.ws.steer,
                                           e.md.dm.d_model, e.mv.dm.vocab, e.mlp ? e.ws.ubias : nullptr,
                                           e.nbias);
}

// Final-norm rows (debug read of the verifier's hidden states).
template <typename TW>
__global__ void k_rmsnorm_rows(const float* X, int d, const TW* gamma, float eps, float* Y) {
    __shared__ float red[4];
    int r = blockIdx.x;
    const float* x = X + (size_t)r * d;
    float ss = 0.0f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) ss += x[i] * x[i];
    ss = wave_sum(ss);
    int lane = threadIdx.x & 63, wave = threadIdx.x / 64;
    if (lane == 0) red[wave] = ss;
    __syncthreads();
    float tot = 0.0f;
    for (int w = 0; w < (int)(blockDim.x / 64); ++w) tot += red[w];
    float sc = rsqrtf(tot / (float)d + eps);
    for (int i = threadIdx.x; i < d; i += blockDim.x) Y[(size_t)r * d + i] = x[i] * sc * load_scalar<TW>(gamma, i);
}

void launch_rmsnorm_rows(hipStream_t s, const float* X, int rows, int d, const void* gamma, bool bf16, float eps,
                         float* Y) {
    if (bf16) k_rmsnorm_rows<uint16_t><<<rows, 256, 0, s>>>(X, d, (const uint16_t*)gamma, eps, Y);
    else k_rmsnorm_rows<float><<<rows, 256, 0, s>>>(X, d, (const float*)gamma, eps, Y);
}

__global__ void k_set_flag(int32_t* f, int v) { *f = v; }
void launch_set_flag(hipStream_t s, int32_t* flag, int v) { k_set_flag<<<1, 1, 0, s>>>(flag, v); }

// ===========================================================================
// Training-objective forward: per-target KL divergence between the verifier and the steered
// drafter (one kernel per operation; see sd2_train_loss).
// ===========================================================================
// Length of the one sequence and the zero row that targets without an earlier steering source read.
__global__ void k_loss_setup(int32_t* len, int n, float* zero_row, int d) {
    if (blockIdx.x == 0 && threadIdx.x == 0) *len = n;
    for (int i = threadIdx.x; i < d; i += blockDim.x) zero_row[i] = 0.0f;
}

// Source row of every drafter input row of a chunk: the verifier position p - delta[p + 1] whose
// final-norm hidden state gives the steering of target p + 1, or the zero row (before the sequence
// start, and for offsets outside 1..k).
__global__ void k_loss_map(int32_t* src, const int32_t* deltas, int pos0, int rows, int n, int k, int zero_row) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const int p = pos0 + r;
    int q = -1;
    if (p < n - 1) {
        const int d = deltas[p + 1];
        if (d >= 1 && d <= k) q = p - d;
    }
    src[r] = q >= 0 ? q : zero_row;
}

// KL(p_V || p_D) of one row of verifier logits A and drafter logits B (temperature 1), three
// passes over the vocabulary: maxima, normalisers, then sum_v p_V (log p_V - log p_D).
__global__ __launch_bounds__(256) void k_kl_rows(const float* A, const float* B, int V, int pos0, int n,
                                                 float* out_kl) {
    __shared__ float red[2][4];
    const int r = blockIdx.x, tau = pos0 + r + 1;
    if (tau > n - 1) return;
    const float* a = A + (size_t)r * V;
    const float* b = B + (size_t)r * V;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    auto block2 = [&](float& x, float& y, bool is_max) {
        x = is_max ? wave_max(x) : wave_sum(x);
        y = is_max ? wave_max(y) : wave_sum(y);
        __syncthreads();
        if (lane == 0) {
            red[0][wave] = x;
            red[1][wave] = y;
        }
        __syncthreads();
        float x0 = red[0][0], y0 = red[1][0];
        for (int w = 1; w < 4; ++w) {
            x0 = is_max ? fmaxf(x0, red[0][w]) : x0 + red[0][w];
            y0 = is_max ? fmaxf(y0, red[1][w]) : y0 + red[1][w];
        }
        x = x0;
        y = y0;
    };
    float ma = -INFINITY, mb = -INFINITY;
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        ma = fmaxf(ma, a[v]);
        mb = fmaxf(mb, b[v]);
    }
    block2(ma, mb, true);
    float za = 0.0f, zb = 0.0f;
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        za += expf(a[v] - ma);
        zb += expf(b[v] - mb);
    }
    block2(za, zb, false);
    const float lsa = ma + logf(za), lsb = mb + logf(zb);
    float kl = 0.0f, unused = 0.0f;
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        const float lpa = a[v] - lsa, lpb = b[v] - lsb;
        kl += expf(lpa) * (lpa - lpb);
    }
    block2(kl, unused, false);
    if (threadIdx.x == 0) out_kl[tau] = kl;
}

// out_kl[0] = 0 and the mean of out_kl[1 .. n-1].
__global__ __launch_bounds__(256) void k_loss_finish(float* out_kl, int n, float* out_loss) {
    __shared__ float red[4];
    float s = 0.0f;
    for (int i = 1 + threadIdx.x; i < n; i += blockDim.x) s += out_kl[i];
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        out_kl[0] = 0.0f;
        *out_loss = (red[0] + red[1] + red[2] + red[3]) / (float)(n - 1);
    }
}

void launch_train_loss(hipStream_t s, Engine& e, const int32_t* tokens, const int32_t* deltas, int n, int chunk,
                       const LossScratch& w, float* out_kl, float* out_loss) {
    const int dV = e.mv.dm.d_model, dD = e.md.dm.d_model, V = e.mv.dm.vocab;
    const int nchunks = (n - 1 + chunk - 1) / chunk;
    const int zero_row = nchunks * chunk;
    k_loss_setup<<<1, 256, 0, s>>>(w.len, n, w.hf + (size_t)zero_row * dV, dV);
    for (int c = 0; c < nchunks; ++c) {
        // verifier over the chunk's positions: its final-norm hidden rows (steering sources) and logits
        launch_plan_embed(s, e, e.mv, kPlanPrefill, c, chunk, tokens, w.len, n, chunk);
        for (int l = 0; l < e.mv.dm.n_layers; ++l) launch_layer(s, e, e.mv, l, chunk, chunk);
        launch_rmsnorm_rows(s, e.mv.x, chunk, dV, e.mv.final_norm, e.bf16, e.mv.dm.rms_eps,
                            w.hf + (size_t)c * chunk * dV);
        launch_lm_head(e, e.mv, chunk, w.lv, nullptr);
        // steering of every target of the chunk: W_s applied to its source row
        k_loss_map<<<(chunk + 255) / 256, 256, 0, s>>>(w.src, deltas, c * chunk, chunk, n, e.cfg.k, zero_row);
        if (e.bf16) {
            WsCall p = ws_base(e, e.mv);
            p.X = w.hf; p.in_map = w.src; p.M = chunk; p.K = dV;
            p.W[0] = e.w_steer; p.seg_rows[0] = dD; p.nseg = 1; p.mode = kEpiStore;
            p.Y = w.srow; p.ldy = dD;
            launch_wsgemv(&e, s, p);
        } else {
            const void* ws[1] = {e.w_steer};
            int rws[1] = {dD};
            launch_gemv(&e, s, false, w.hf, w.src, chunk, dV, nullptr, 0.f, ws, rws, 1, kEpiStore, w.srow, dD,
                        nullptr);
        }
        // drafter over the same positions, each input embedding plus its target's steering
        launch_plan_embed(s, e, e.md, kPlanPrefill, c, chunk, tokens, w.len, n, chunk, w.srow);
        for (int l = 0; l < e.md.dm.n_layers; ++l) launch_layer(s, e, e.md, l, chunk, chunk);
        launch_lm_head(e, e.md, chunk, w.ld, nullptr);
        k_kl_rows<<<chunk, 256, 0, s>>>(w.lv, w.ld, V, c * chunk, n, out_kl);
    }
    k_loss_finish<<<1, 256, 0, s>>>(out_kl, n, out_loss);
}

}  // namespace sd2
