// Host side of the SD^2 engine: argument checks, workspace carving, the round's kernel
// sequence (recorded once into a HIP graph and replayed), prefill, and the C ABI.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>

#include "engine.h"

using namespace sd2;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Carver {
    char* base;
    size_t off = 0;
    template <typename T>
    T* take(size_t count) {
        off = align_up(off);
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

bool dims_ok(const sd2_dims& d) {
    if (d.n_layers < 1 || d.n_layers > 128 || d.d_model < 64 || d.n_heads < 1 || d.n_kv_heads < 1 ||
        d.d_ff < 64 || d.vocab < 2)
        return false;
    if (d.d_model % d.n_heads || d.n_heads % d.n_kv_heads) return false;
    int hd = d.d_model / d.n_heads;
    if (hd != 32 && hd != 64 && hd != 128) return false;
    if (d.d_model % 64 || (d.n_heads * hd) % 64 || d.d_ff % 64) return false;
    // the residual row is at most 16384 wide; d_ff has no further limit for bf16 weights (the
    // projection kernels split K into ranges); f32 weights: see config_ok
    if (d.d_model > 16384 || d.d_ff > 65536) return false;
    if (!(d.rope_theta > 0.f) || !(d.rms_eps >= 0.f)) return false;
    return true;
}

bool bf16_dims_ok(const sd2_dims& d) {
    // the bf16 projection kernel splits K into multiples of 256 and N into 16-row tiles;
    // attention kernels exist for head dims 32, 64 and 128
    int hd = d.d_model / d.n_heads;
    return d.d_model % 256 == 0 && (d.n_heads * hd) % 256 == 0 && d.d_ff % 256 == 0 && d.vocab % 16 == 0 &&
           (hd == 32 || hd == 64 || hd == 128);
}

bool mlp_form(const sd2_config& c);

bool config_ok(const sd2_config* c) {
    if (!c) return false;
    if (!dims_ok(c->verifier) || !dims_ok(c->drafter)) return false;
    if (c->dtype == SD2_BF16 && (!bf16_dims_ok(c->verifier) || !bf16_dims_ok(c->drafter))) return false;
    if (c->verifier.vocab != c->drafter.vocab) return false;
    if (c->dtype != SD2_F32 && c->dtype != SD2_BF16) return false;
    // f32 weights use the vector projection kernel, which stages a whole input row in 64 KB of LDS
    if (c->dtype == SD2_F32 && (c->verifier.d_ff > 16384 || c->drafter.d_ff > 16384)) return false;
    if (c->k < 1 || c->k > kMaxK) return false;
    if (c->max_batch < 1 || c->max_batch > 256) return false;
    if (c->max_new_tokens < 1) return false;
    if (c->max_seq_len < c->k + 3 || c->max_seq_len > 8192) return false;  // the capacity the kernels are tested to
    if (!(c->temperature >= 0.f) || c->temperature > 1e4f) return false;
    if (c->steering != SD2_STEER_INPUT && c->steering != SD2_STEER_MLP && c->steering != SD2_STEER_MLP_OUT &&
        c->steering != SD2_STEER_NONE && c->steering != SD2_STEER_MLP_COND)
        return false;
    if (c->steering == SD2_STEER_MLP_COND && (c->cond_rank < 16 || c->cond_rank > 4096 || c->cond_rank % 16))
        return false;
    if (mlp_form(*c)) {
        // the low tap is block 3; a steering projection runs on the MFMA kernel when its K is a
        // multiple of 256 (bf16), else on the vector kernel, which stages a K row of at most 16384
        const int dV = c->verifier.d_model;
        if (c->verifier.n_layers < 3) return false;
        if (3 * dV > 16384 && !(c->dtype == SD2_BF16 && (3 * dV) % 256 == 0)) return false;
        if (dV > 16384 && !(c->dtype == SD2_BF16 && dV % 256 == 0)) return false;
    }
    return true;
}

// MLP steering forms (taps, W_hml, LayerNorm, biases in the drafter's MLPs)
bool mlp_form(const sd2_config& c) {
    return c.steering == SD2_STEER_MLP || c.steering == SD2_STEER_MLP_OUT || c.steering == SD2_STEER_MLP_COND;
}

// MLP steering: bias values per sequence (per-layer up-projection biases, or one after-MLP bias)
int bias_len(const sd2_config& c) {
    if (c.steering == SD2_STEER_MLP_COND) return c.drafter.n_layers * c.cond_rank;  // the g parts V_l^g g
    return c.steering == SD2_STEER_MLP ? c.drafter.n_layers * c.drafter.d_ff : c.drafter.d_model;
}

int max_rows(const sd2_config& c) {
    int B = c.max_batch;
    return std::max(std::max(B * (c.k + 1), 2 * B), kPrefillRows);
}

void model_dims(ModelDev* m, const sd2_dims& d) {
    m->dm = d;
    m->hd = d.d_model / d.n_heads;
    m->qkv_dim = (d.n_heads + 2 * d.n_kv_heads) * m->hd;
}

}  // namespace

namespace sd2 {

size_t carve(const sd2_config& c, char* base, Workspace* ws, ModelDev* mv, ModelDev* md, int* maxm_out,
             MkState* mk) {
    Carver cv{base};
    int B = c.max_batch, k = c.k, cap = c.max_seq_len, V = c.verifier.vocab;
    int maxm = max_rows(c);
    if (maxm_out) *maxm_out = maxm;
    ModelDev tv, td;
    model_dims(&tv, c.verifier);
    model_dims(&td, c.drafter);
    ModelDev* ms[2] = {mv ? mv : &tv, md ? md : &td};
    if (mv) model_dims(mv, c.verifier);
    if (md) model_dims(md, c.drafter);
    Workspace w{};
    w.t = cv.take<int32_t>(B);
    w.len_v = cv.take<int32_t>(B);
    w.len_d = cv.take<int32_t>(B);
    w.produced = cv.take<int32_t>(B);
    w.done = cv.take<int32_t>(B);
    w.hist = cv.take<int32_t>((size_t)B * cap);
    w.steer = cv.take<float>((size_t)B * c.drafter.d_model);
    w.hcap = cv.take<float>((size_t)B * c.verifier.d_model);
    w.hcap_ss = cv.take<float>((size_t)B * (c.verifier.d_model / 16));
    w.row_pos = cv.take<int32_t>(maxm);
    w.row_seq = cv.take<int32_t>(maxm);
    w.lm_map_d = cv.take<int32_t>((size_t)k * 2 * B);
    w.steer_map = cv.take<int32_t>(B);
    w.ident_map = cv.take<int32_t>(2 * (size_t)B);
    int qkv = std::max(ms[0]->qkv_dim, ms[1]->qkv_dim);
    int att = std::max(c.verifier.n_heads * ms[0]->hd, c.drafter.n_heads * ms[1]->hd);
    int ff = std::max(c.verifier.d_ff, c.drafter.d_ff);
    w.qkv = cv.take<float>((size_t)maxm * qkv);
    w.attn = cv.take<float>((size_t)maxm * att);
    w.ffh = cv.take<float>((size_t)maxm * ff);
    w.logits_v = cv.take<float>((size_t)B * (k + 1) * V);
    w.logits_d = cv.take<float>((size_t)B * k * V);
    w.hidden_dbg = cv.take<float>((size_t)B * (k + 1) * c.verifier.d_model);
    w.part = cv.take<VPart>((size_t)B * (2 * k + 1) * kVocabChunks);
    w.lse_v = cv.take<float>((size_t)B * (k + 1));
    w.lse_d = cv.take<float>((size_t)B * k);
    w.argmax_v = cv.take<int32_t>((size_t)B * (k + 1));
    w.drafts = cv.take<int32_t>((size_t)B * k);
    w.own_drafts = cv.take<int32_t>((size_t)B * k);
    w.n_eff = cv.take<int32_t>(B);
    w.own_n = cv.take<int32_t>(B);
    w.own_y = cv.take<int32_t>(B);
    w.forced = cv.take<int32_t>((size_t)B * (k + 2));
    w.forced_on = cv.take<int32_t>(1);
    // projection split-K partials: the largest tiles*S*256*subs over every projection shape
    {
        size_t pmax = 0, pg_cnt = 0;
        const sd2_dims* dd[2] = {&c.verifier, &c.drafter};
        int mmax = std::min(maxm, 16);
        for (int i = 0; i < 2; ++i) {
            const sd2_dims& d = *dd[i];
            int hd = d.d_model / d.n_heads;
            int shapes[6][3] = {{(d.n_heads + 2 * d.n_kv_heads) * hd, d.d_model, kEpiQkv},
                                {d.d_model, d.n_heads * hd, kEpiAdd},
                                {d.d_ff, d.d_model, kEpiSwiglu},
                                {d.d_model, d.d_ff, kEpiAdd},
                                {d.vocab, d.d_model, kEpiStore},
                                {c.drafter.d_model, c.verifier.d_model, kEpiStore}};
            for (int mm = 1; mm <= mmax; ++mm)
                for (auto& sh : shapes) {
                    WsPlan p = ws_plan(mm, sh[0], sh[1], sh[2]);
                    size_t subs = sh[2] == kEpiSwiglu ? 2 : 1;
                    if (p.S > 1) pmax = std::max(pmax, (size_t)p.tiles * p.S * 256 * subs);
                }
        }
        if (mlp_form(c)) {
            // W_hml (d_V x 3 d_V) and W_s (bias values x d_V) projections; the conditional bias's
            // V^f (R x d_D) and U (d_ff x R) on the drafter's rows
            const int R = c.steering == SD2_STEER_MLP_COND ? c.cond_rank : 0;
            int mshapes[4][3] = {{c.verifier.d_model, 3 * c.verifier.d_model, std::min(B, 16)},
                                 {bias_len(c), c.verifier.d_model, std::min(B, 16)},
                                 {R, c.drafter.d_model, std::min(2 * B, 16)},
                                 {c.drafter.d_ff, R, std::min(2 * B, 16)}};
            for (auto& sh : mshapes)
                for (int mm = 1; sh[0] > 0 && mm <= sh[2]; ++mm) {
                    WsPlan p = ws_plan(mm, sh[0], sh[1], kEpiStore);
                    if (p.S > 1) pmax = std::max(pmax, (size_t)p.tiles * p.S * 256);
                }
        }
        // many-row GEMM with K ranges: [tile][m block][range][subs][4 x 256] partials.  Besides the
        // models' projections: W_s over many rows (the training-objective forward) and the MLP
        // steering projections at batches above 16 rows
        const int R = c.steering == SD2_STEER_MLP_COND ? c.cond_rank : 0;
        const bool mf = mlp_form(c);
        for (int i = 0; i < 2; ++i) {
            const sd2_dims& d = *dd[i];
            int hd = d.d_model / d.n_heads;
            int shapes[10][3] = {{(d.n_heads + 2 * d.n_kv_heads) * hd, d.d_model, 1},
                                 {d.d_model, d.n_heads * hd, 1},
                                 {d.d_ff, d.d_model, 2},
                                 {d.d_model, d.d_ff, 1},
                                 {d.vocab, d.d_model, 1},
                                 {c.drafter.d_model, c.verifier.d_model, 1},
                                 {mf ? c.verifier.d_model : 0, 3 * c.verifier.d_model, 1},
                                 {mf ? bias_len(c) : 0, c.verifier.d_model, 1},
                                 {R, c.drafter.d_model, 1},
                                 {R ? c.drafter.d_ff : 0, R, 1}};
            // the split depends on the rows only through their number of 64-row blocks
            for (int nbm = 1; nbm <= (maxm + 63) / 64; ++nbm)
                for (auto& sh : shapes) {
                    if (sh[0] <= 0) continue;
                    int S = pg_split(nbm * 64, sh[0], sh[1], sh[2]);
                    size_t nblkm = (size_t)nbm;
                    if (S > 1) {
                        pmax = std::max(pmax, nblkm * (sh[0] / 16) * S * sh[2] * 1024);
                        pg_cnt = std::max(pg_cnt, nblkm * (sh[0] / 16));
                    }
                }
        }
        w.ws_part = cv.take<float>(std::max<size_t>(pmax, 1));
        w.ws_part_n = std::max<size_t>(pmax, 1);
        size_t tmax = (size_t)std::max(c.verifier.vocab, c.drafter.vocab) / 16 + 1;
        for (int i = 0; i < 2; ++i)
            tmax = std::max(tmax, (size_t)std::max(dd[i]->d_ff, dd[i]->d_model) / 16 + 1);
        if (mlp_form(c)) tmax = std::max(tmax, (size_t)bias_len(c) / 16 + 1);
        tmax = std::max(tmax, pg_cnt);
        w.ws_cnt = cv.take<int32_t>(tmax);
        w.ws_cnt_n = tmax;
    }
    {
        size_t amax = 0;
        const sd2_dims* dd[2] = {&c.verifier, &c.drafter};
        for (int i = 0; i < 2; ++i) {
            int hd = dd[i]->d_model / dd[i]->n_heads;
            amax = std::max(amax, (size_t)maxm * dd[i]->n_heads * attn_nsplit(cap) * (hd + 2));
        }
        w.attn_part = cv.take<float>(amax);
        // arrival counters: the largest split-free grid of any launch shape
        size_t gmax = 1;
        for (int i = 0; i < 2; ++i) {
            const sd2_dims& d = *dd[i];
            gmax = std::max(gmax, attn_groups(2 * B, 2, d.n_heads, d.n_kv_heads));
            gmax = std::max(gmax, attn_groups(B, 1, d.n_heads, d.n_kv_heads));
            gmax = std::max(gmax, attn_groups(B * (c.k + 1), c.k + 1, d.n_heads, d.n_kv_heads));
            for (int nseq = 1; nseq <= B; ++nseq) {
                int rps = std::max(1, kPrefillRows / nseq);
                gmax = std::max(gmax, attn_groups(nseq * rps, rps, d.n_heads, d.n_kv_heads));
            }
        }
        w.attn_cnt = cv.take<int32_t>(gmax);
        w.nonfinite = cv.take<int32_t>(4);
        w.attn_cnt_n = gmax;
    }
    if (mlp_form(c)) {
        const size_t dV = c.verifier.d_model;
        w.taps = cv.take<float>(3 * (size_t)maxm * dV);
        w.tapsel = cv.take<float>((size_t)B * 3 * dV);
        w.gsteer = cv.take<float>((size_t)B * dV);
        w.ubias = cv.take<float>((size_t)B * bias_len(c));
        if (c.steering == SD2_STEER_MLP_COND) {
            w.cond_h = cv.take<float>((size_t)2 * B * c.cond_rank);
            w.cond_b = cv.take<float>((size_t)2 * B * c.drafter.d_ff);
        }
    }
    for (int i = 0; i < 2; ++i) {
        ModelDev* m = ms[i];
        const sd2_dims& d = m->dm;
        size_t kv = (size_t)d.n_layers * B * d.n_kv_heads * cap * m->hd;
        m->kc = cv.take<float>(kv);
        m->vc = cv.take<float>(kv);
        m->rope_cos = cv.take<float>((size_t)cap * (m->hd / 2));
        m->rope_sin = cv.take<float>((size_t)cap * (m->hd / 2));
        m->x = cv.take<float>((size_t)maxm * d.d_model);
        m->ss = cv.take<float>((size_t)maxm * (d.d_model / 16));
    }
    // persistent round-program path: phase lists, activation arena, barrier and hand-off state
    {
        MkState st{};
        st.max_batch = mk_max_batch(c);
        if (st.max_batch > 0) {
            st.prog_cap = mk_phase_count(c);
            st.prog = cv.take<MkPhase>((size_t)st.prog_cap);
            st.arena_bytes = mk_arena_bytes(c, st.max_batch);
            st.arena = cv.take<char>(st.arena_bytes);
            st.bar = cv.take<int32_t>(kMkBarInts);
            st.err = cv.take<int32_t>(64);
            st.qc = cv.take<int32_t>((size_t)2 * kMkQcLines * kMkLine);
            st.cnt = cv.take<int32_t>(mk_counter_ints(c));
            st.dummy = cv.take<uint16_t>(512);
            st.ones = cv.take<uint16_t>(kMkMaxKR);
            st.trace = cv.take<int64_t>((size_t)kMkMaxLaunch * kMkTracePhases);
        }
        if (mk) *mk = st;
    }
    if (ws) *ws = w;
    return align_up(cv.off);
}

}  // namespace sd2

namespace sd2 {

void prof_begin(Engine* e, int cls, double bytes) {
    if (!e || !e->prof_on || e->prof_n >= kProfMax) return;
    ProfEntry& p = e->prof[e->prof_n];
    if (!p.a) return;
    p.cls = cls;
    p.bytes = bytes;
    (void)hipEventRecord(p.a, e->stream);
}

ProfEntry* prof_slot(Engine* e, int cls, double bytes) {
    if (!e || !e->prof_on || e->prof_n >= kProfMax) return nullptr;
    ProfEntry& p = e->prof[e->prof_n];
    if (!p.a) return nullptr;
    p.cls = cls;
    p.bytes = bytes;
    return &p;
}

void prof_commit(Engine* e) {
    if (e && e->prof_on && e->prof_n < kProfMax) ++e->prof_n;
}

void prof_end(Engine* e) {
    if (!e || !e->prof_on || e->prof_n >= kProfMax) return;
    ProfEntry& p = e->prof[e->prof_n];
    if (!p.a) return;
    (void)hipEventRecord(p.b, e->stream);
    ++e->prof_n;
}

}  // namespace sd2

namespace {

sd2_status hip_fail(Engine* e, hipError_t err, const char* where) {
    snprintf(e->err, sizeof(e->err), "%s: %s", where, hipGetErrorString(err));
    return SD2_ERR_HIP;
}

sd2_status check_launch(Engine* e, const char* where) {
    if (e->launch_err != hipSuccess) {
        hipError_t err = e->launch_err;
        e->launch_err = hipSuccess;
        return hip_fail(e, err, where);
    }
    if (e->bad_launch) {
        snprintf(e->err, sizeof(e->err), "%s: no projection kernel instance for a shape", where);
        return SD2_ERR_UNSUPPORTED;
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(e, err, where);
    return SD2_OK;
}

// The whole round, as a fixed sequence of kernels (no host decisions).
void enqueue_round(Engine& e, int32_t* out_tokens, int32_t* out_counts) {
    hipStream_t s = e.stream;
    e.prof_n = 0;
    int B = e.batch, k = e.cfg.k;
    if (e.mk.active) {
        // one persistent launch per drafter step and one for the verifier block
        for (int j = 1; j <= k; ++j) {
            hipError_t err = mk_launch(e, j);
            if (err != hipSuccess) { e.launch_err = err; return; }
            launch_draft_pick(s, e, j);
        }
        hipError_t err = mk_launch(e, 0);
        if (err != hipSuccess) { e.launch_err = err; return; }
        launch_verify_decide(s, e, out_tokens, out_counts);
        if (e.mlp) launch_mlp_steer(e, e.mk.tap_x, e.ws.steer_map, B);
        else if (e.w_steer) launch_steer(e, e.mk.final_x, e.mk.final_ss, e.ws.steer_map, B);
        return;
    }
    const int ub_ld = e.nbias;
    for (int j = 1; j <= k; ++j) {
        int rows = j == 1 ? 2 * B : B;
        launch_plan_embed(s, e, e.md, j == 1 ? kPlanDraft1 : kPlanDraftJ, j, rows, nullptr, nullptr, 0, 1);
        for (int l = 0; l < e.md.dm.n_layers; ++l) {
            if (e.cond) {
                // this layer's bias of every row, from the row's residual as it enters the layer
                launch_cond_bias(s, e, l, rows);
                launch_layer(s, e, e.md, l, rows, j == 1 ? 2 : 1, e.ws.cond_b, e.md.dm.d_ff, false,
                             e.ws.ident_map);
                continue;
            }
            launch_layer(s, e, e.md, l, rows, j == 1 ? 2 : 1,
                         !e.mlp ? nullptr : e.ws.ubias + (e.bias_after ? 0 : (size_t)l * e.md.dm.d_ff), ub_ld,
                         e.bias_after);
        }
        launch_lm_head(e, e.md, rows, e.ws.logits_d, e.ws.lm_map_d + (size_t)(j - 1) * 2 * e.cfg.max_batch);
        launch_draft_pick(s, e, j);
    }
    int rows = B * (k + 1);
    launch_plan_embed(s, e, e.mv, kPlanVerify, 0, rows, nullptr, nullptr, 0, 1);
    for (int l = 0; l < e.mv.dm.n_layers; ++l) {
        launch_layer(s, e, e.mv, l, rows, k + 1);
        if (e.mlp) launch_tap_copy(s, e, l, rows);
    }
    launch_lm_head(e, e.mv, rows, e.ws.logits_v, nullptr);
    launch_verify_decide(s, e, out_tokens, out_counts);
    if (e.mlp) {
        const size_t slot = (size_t)e.maxm * e.mv.dm.d_model;
        const float* src[3] = {e.ws.taps, e.ws.taps + slot, e.ws.taps + 2 * slot};
        launch_mlp_steer(e, src, e.ws.steer_map, B);
    } else if (e.w_steer) {
        launch_steer(e, e.mv.x, e.mv.ss, e.ws.steer_map, B);
    }
}

void drop_graph(Engine& e) {
    if (e.graph_exec) (void)hipGraphExecDestroy(e.graph_exec);
    if (e.graph) (void)hipGraphDestroy(e.graph);
    e.graph_exec = nullptr;
    e.graph = nullptr;
}

sd2_status run_round(Engine* e, int32_t* out_tokens, int32_t* out_counts) {
    // Replay the recorded round when the shape and output buffers are unchanged.  Profiled rounds
    // are launched eagerly: HIP events recorded inside a captured graph cannot be timed.
    if (!e->use_graph || e->prof_on || e->mk.active) {
        enqueue_round(*e, out_tokens, out_counts);
        return check_launch(e, "round");
    }
    if (!e->graph_exec || e->graph_batch != e->batch || e->graph_out_tokens != out_tokens ||
        e->graph_out_counts != out_counts) {
        drop_graph(*e);
        hipError_t err = hipStreamBeginCapture(e->stream, hipStreamCaptureModeThreadLocal);
        if (err != hipSuccess) return hip_fail(e, err, "hipStreamBeginCapture");
        enqueue_round(*e, out_tokens, out_counts);
        err = hipStreamEndCapture(e->stream, &e->graph);
        if (err != hipSuccess) return hip_fail(e, err, "hipStreamEndCapture");
        err = hipGraphInstantiate(&e->graph_exec, e->graph, nullptr, nullptr, 0);
        if (err != hipSuccess) return hip_fail(e, err, "hipGraphInstantiate");
        e->graph_batch = e->batch;
        e->graph_out_tokens = out_tokens;
        e->graph_out_counts = out_counts;
    }
    hipError_t err = hipGraphLaunch(e->graph_exec, e->stream);
    if (err != hipSuccess) return hip_fail(e, err, "hipGraphLaunch");
    return SD2_OK;
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// Workspace that needs no allocation (sd2_create_noalloc): a static device array, one copy per
// GPU, held from the library's load until the process ends.  In host code `scratch` names a
// host-side stand-in, not the device copy: its device address on each GPU comes from
// hipGetSymbolAddress (once per device, with that device current), and only that address is
// ever handed to kernels.  One handle at a time per device uses it; the handle's host state
// lives in the same per-device slot, so creating it allocates nothing on host or device.
// ---------------------------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

namespace {

constexpr int kStaticMaxDevices = 64;

struct StaticSlot {
    void* ptr;    // device address of `scratch` on this device (null until first looked up)
    bool live;    // a handle created by sd2_create_noalloc uses it
    Engine engine;
};
StaticSlot g_static[kStaticMaxDevices];
std::mutex g_static_mu;

// Clears n bytes (a multiple of 16) with vector stores: a kernel rather than hipMemsetAsync, so
// that a caller may capture the creation into a graph.
__global__ void k_zero16(uint4* p, size_t n16) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) p[i] = make_uint4(0, 0, 0, 0);
}

}  // namespace

extern "C" {

size_t sd2_workspace_bytes(const sd2_config* cfg) {
    if (!config_ok(cfg)) return 0;
    return carve(*cfg, nullptr, nullptr, nullptr, nullptr, nullptr);
}

const char* sd2_status_string(sd2_status s) {
    switch (s) {
        case SD2_OK: return "ok";
        case SD2_ERR_INVALID_ARG: return "invalid argument";
        case SD2_ERR_CAPACITY: return "capacity exceeded (max_seq_len, or sd2_create_noalloc's static workspace)";
        case SD2_ERR_STATE: return "invalid state (prefill first)";
        case SD2_ERR_HIP: return "HIP runtime error";
        case SD2_ERR_UNSUPPORTED: return "unsupported";
        default: return "unknown status";
    }
}

const char* sd2_last_error(sd2_handle_t h) {
    if (!h) return "";
    return reinterpret_cast<Engine*>(h)->err;
}

static bool aligned16(const void* p) { return p && ((uintptr_t)p % 16) == 0; }

static bool weights_ok(const sd2_weights* w, const sd2_dims& d) {
    if (!w || !aligned16(w->embed) || !w->layers || !aligned16(w->final_norm) || !aligned16(w->lm_head)) return false;
    for (int i = 0; i < d.n_layers * 9; ++i)
        if (!aligned16(w->layers[i])) return false;
    return true;
}

// slot: the per-device static slot whose Engine and workspace to use (sd2_create_noalloc), or null
static sd2_status create_impl(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                              const void* w_steer, const sd2_mlp_steering* mlp, void* workspace,
                              size_t workspace_bytes, void* hip_stream, sd2_handle_t* out,
                              StaticSlot* slot = nullptr) {
    if (!out) return SD2_ERR_INVALID_ARG;
    *out = nullptr;
    if (!config_ok(cfg)) return SD2_ERR_INVALID_ARG;
    if (mlp_form(*cfg) != (mlp != nullptr)) return SD2_ERR_INVALID_ARG;
    if (mlp && (!aligned16(mlp->w_hml) || !aligned16(mlp->ln_gain) || !aligned16(mlp->ln_bias) ||
                !(mlp->ln_eps >= 0.f)))
        return SD2_ERR_INVALID_ARG;
    if (!weights_ok(verifier, cfg->verifier) || !weights_ok(drafter, cfg->drafter)) return SD2_ERR_INVALID_ARG;
    const bool unsteered = cfg->steering == SD2_STEER_NONE;
    if (!unsteered && !aligned16(w_steer)) return SD2_ERR_INVALID_ARG;
    if (!workspace || ((uintptr_t)workspace % kAlign) != 0) return SD2_ERR_INVALID_ARG;
    size_t need = sd2_workspace_bytes(cfg);
    if (workspace_bytes < need) return SD2_ERR_INVALID_ARG;
    // the kernels are built for gfx950 with XNACK (page-fault replay) off, MI355X's default mode
    {
        int dev = 0;
        hipDeviceProp_t prop;
        if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
            return SD2_ERR_HIP;
        if (strncmp(prop.gcnArchName, "gfx950", 6) != 0 || strstr(prop.gcnArchName, "xnack+") != nullptr)
            return SD2_ERR_UNSUPPORTED;
    }
    Engine* e = nullptr;
    if (slot) {
        slot->engine = Engine{};
        e = &slot->engine;
        e->static_slot = true;
    } else {
        e = new (std::nothrow) Engine();
        if (!e) return SD2_ERR_INVALID_ARG;
    }
    e->cfg = *cfg;
    e->cap = cfg->max_seq_len;
    e->bf16 = cfg->dtype == SD2_BF16;
    e->stream = (hipStream_t)hip_stream;
    e->w_steer = unsteered ? nullptr : w_steer;
    e->mlp = mlp != nullptr;
    e->bias_after = cfg->steering == SD2_STEER_MLP_OUT;
    e->nbias = bias_len(*cfg);
    if (mlp) {
        e->cond = cfg->steering == SD2_STEER_MLP_COND;
        if (e->cond && (!aligned16(mlp->w_cf) || !aligned16(mlp->w_cu))) {
            if (!slot) delete e;
            return SD2_ERR_INVALID_ARG;
        }
        e->w_cf = mlp->w_cf;
        e->w_cu = mlp->w_cu;
        e->w_hml = mlp->w_hml;
        e->ln_gain = mlp->ln_gain;
        e->ln_bias = mlp->ln_bias;
        e->ln_eps = mlp->ln_eps;
    }
    {
        // blocks L-2, floor(L/2) and 3 counted from 1 (high, middle, low)
        const int L = cfg->verifier.n_layers;
        e->tap_layer[0] = L - 3;
        e->tap_layer[1] = L / 2 - 1;
        e->tap_layer[2] = 2;
    }
    // Graph replay needs a capturable (non-null) stream; SD2_NO_GRAPH=1 forces eager launches.
    e->use_graph = hip_stream != nullptr && getenv("SD2_NO_GRAPH") == nullptr;
    carve(*cfg, (char*)workspace, &e->ws, &e->mv, &e->md, &e->maxm, &e->mk);
    const sd2_weights* src[2] = {verifier, drafter};
    ModelDev* dst[2] = {&e->mv, &e->md};
    for (int i = 0; i < 2; ++i) {
        dst[i]->embed = src[i]->embed;
        dst[i]->final_norm = src[i]->final_norm;
        dst[i]->lm_head = src[i]->lm_head;
        for (int j = 0; j < dst[i]->dm.n_layers * 9; ++j) dst[i]->layer[j] = src[i]->layers[j];
    }
    hipError_t err = wsgemv_setup();
    if (err != hipSuccess) {
        sd2_status st = hip_fail(e, err, "hipFuncSetAttribute");
        if (!slot) delete e;
        return st;
    }
    if (slot) {
        // the static workspace keeps the previous handle's contents: clear it with a kernel
        const size_t n16 = (need + 15) / 16;
        k_zero16<<<(unsigned)std::min<size_t>(4096, (n16 + 255) / 256), 256, 0, e->stream>>>((uint4*)workspace, n16);
        err = hipGetLastError();
    } else {
        err = hipMemsetAsync(workspace, 0, need, e->stream);
    }
    if (err != hipSuccess) {
        sd2_status st = hip_fail(e, err, slot ? "k_zero16" : "hipMemsetAsync");
        if (!slot) delete e;
        return st;
    }
    launch_rope_table(e->stream, e->mv, e->cap);
    launch_rope_table(e->stream, e->md, e->cap);
    launch_init_maps(e->stream, *e);
    mk_init_buffers(*e);
    sd2_status st = check_launch(e, "create");
    if (st != SD2_OK) {
        if (!slot) delete e;
        return st;
    }
    *out = reinterpret_cast<sd2_handle_t>(e);
    return SD2_OK;
}

sd2_status sd2_create(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                      const void* w_steer, void* workspace, size_t workspace_bytes, void* hip_stream,
                      sd2_handle_t* out) {
    return create_impl(cfg, verifier, drafter, w_steer, nullptr, workspace, workspace_bytes, hip_stream, out);
}

// Training-objective forward: buffers for sequences of n tokens in chunks of `chunk` positions.
static size_t loss_carve(const sd2_config& c, int n, int chunk, char* base, LossScratch* out) {
    const int nchunks = (n - 1 + chunk - 1) / chunk;
    const size_t V = c.verifier.vocab, dV = c.verifier.d_model, dD = c.drafter.d_model;
    size_t off = 0;
    auto take = [&](size_t bytes) -> char* {
        char* p = base ? base + off : nullptr;
        off += (bytes + kAlign - 1) / kAlign * kAlign;
        return p;
    };
    LossScratch w{};
    w.lv = (float*)take(sizeof(float) * chunk * V);
    w.ld = (float*)take(sizeof(float) * chunk * V);
    w.hf = (float*)take(sizeof(float) * ((size_t)nchunks * chunk + 1) * dV);
    w.srow = (float*)take(sizeof(float) * chunk * dD);
    w.src = (int32_t*)take(sizeof(int32_t) * chunk);
    w.len = (int32_t*)take(sizeof(int32_t));
    if (out) *out = w;
    return off;
}

size_t sd2_train_loss_scratch_bytes(const sd2_config* cfg, int32_t max_len, int32_t rows_per_chunk) {
    if (!config_ok(cfg) || cfg->steering != SD2_STEER_INPUT) return 0;
    if (max_len < 2 || max_len > cfg->max_seq_len || rows_per_chunk < 1 || rows_per_chunk > kPrefillRows) return 0;
    return loss_carve(*cfg, max_len, rows_per_chunk, nullptr, nullptr);
}

sd2_status sd2_train_loss(sd2_handle_t h, const int32_t* tokens, const int32_t* deltas, int32_t n,
                          int32_t rows_per_chunk, float* out_kl, float* out_loss, void* scratch,
                          size_t scratch_bytes) {
    if (!h || !tokens || !deltas || !out_kl || !out_loss || !scratch) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (e->cfg.steering != SD2_STEER_INPUT) return SD2_ERR_UNSUPPORTED;
    if (n < 2 || rows_per_chunk < 1 || rows_per_chunk > kPrefillRows) return SD2_ERR_INVALID_ARG;
    if (n > e->cap) return SD2_ERR_CAPACITY;
    if ((uintptr_t)scratch % kAlign || scratch_bytes < loss_carve(e->cfg, n, rows_per_chunk, nullptr, nullptr))
        return SD2_ERR_INVALID_ARG;
    LossScratch w;
    loss_carve(e->cfg, n, rows_per_chunk, (char*)scratch, &w);
    // the forward runs in sequence slot 0 of both caches: the generation state is gone afterwards
    e->batch = 1;
    e->prefilled = false;
    launch_train_loss(e->stream, *e, tokens, deltas, n, rows_per_chunk, w, out_kl, out_loss);
    return check_launch(e, "train_loss");
}

sd2_status sd2_create_noalloc(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                              const void* w_steer, void* hip_stream, sd2_handle_t* out) {
    if (!out) return SD2_ERR_INVALID_ARG;
    *out = nullptr;
    if (!config_ok(cfg) || mlp_form(*cfg)) return SD2_ERR_INVALID_ARG;
    const size_t need = sd2_workspace_bytes(cfg);
    if (need > kStaticWorkspaceBytes) return SD2_ERR_CAPACITY;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return SD2_ERR_HIP;
    if (dev < 0 || dev >= kStaticMaxDevices) return SD2_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_static_mu);
    StaticSlot& slot = g_static[dev];
    if (slot.live) return SD2_ERR_STATE;
    if (!slot.ptr) {
        // the device copy's address on this device (the current one)
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SD2_ERR_HIP;
        slot.ptr = p;
    }
    sd2_status st = create_impl(cfg, verifier, drafter, w_steer, nullptr, slot.ptr, kStaticWorkspaceBytes,
                                hip_stream, out, &slot);
    if (st == SD2_OK) {
        slot.live = true;
        slot.engine.static_device = dev;
    }
    return st;
}

sd2_status sd2_create_mlp(const sd2_config* cfg, const sd2_weights* verifier, const sd2_weights* drafter,
                          const sd2_mlp_steering* steering, void* workspace, size_t workspace_bytes,
                          void* hip_stream, sd2_handle_t* out) {
    if (!steering) {
        if (out) *out = nullptr;
        return SD2_ERR_INVALID_ARG;
    }
    return create_impl(cfg, verifier, drafter, steering->w_s, steering, workspace, workspace_bytes, hip_stream,
                       out);
}

sd2_status sd2_prefill(sd2_handle_t h, int32_t batch, const int32_t* tokens, const int32_t* lens,
                       int32_t max_prompt) {
    if (!h) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (batch < 1 || batch > e->cfg.max_batch || !tokens || !lens || max_prompt < 1) return SD2_ERR_INVALID_ARG;
    if ((int64_t)max_prompt + e->cfg.max_new_tokens + e->cfg.k + 1 > e->cap) return SD2_ERR_CAPACITY;
    hipStream_t s = e->stream;
    e->batch = batch;
    int chunk = std::max(1, std::min(max_prompt - 1, kPrefillRows / batch));
    int rows = batch * chunk;
    int nchunks = max_prompt > 1 ? (max_prompt - 1 + chunk - 1) / chunk : 0;
    hipError_t err = hipMemsetAsync(e->ws.hcap, 0, sizeof(float) * (size_t)batch * e->mv.dm.d_model, s);
    if (err != hipSuccess) return hip_fail(e, err, "hipMemsetAsync");
    for (int c = 0; c < nchunks; ++c) {
        launch_plan_embed(s, *e, e->mv, kPlanPrefill, c, rows, tokens, lens, max_prompt, chunk);
        for (int l = 0; l < e->mv.dm.n_layers; ++l) {
            launch_layer(s, *e, e->mv, l, rows, chunk);
            if (e->mlp) launch_prefill_tap(s, *e, l, rows, lens, max_prompt);
        }
        launch_prefill_capture(s, *e, rows, lens, max_prompt);
    }
    // the first round's steering from position len-2 (a one-token prompt gets none: the finish
    // step below clears it)
    if (e->mlp) launch_mlp_steer(*e, nullptr, nullptr, batch);
    else if (e->w_steer) launch_steer(*e, e->ws.hcap, e->ws.hcap_ss, nullptr, batch);
    for (int c = 0; c < nchunks; ++c) {
        launch_plan_embed(s, *e, e->md, kPlanPrefill, c, rows, tokens, lens, max_prompt, chunk);
        for (int l = 0; l < e->md.dm.n_layers; ++l) launch_layer(s, *e, e->md, l, rows, chunk);
    }
    launch_prefill_finish(s, *e, batch, tokens, lens, max_prompt);
    sd2_status st = check_launch(e, "prefill");
    if (st != SD2_OK) return st;
    // rounds run as persistent launches when the shapes allow it (else as separate kernels)
    mk_build(*e, batch);
    e->prefilled = true;
    return SD2_OK;
}

sd2_status sd2_round(sd2_handle_t h, int32_t* out_tokens, int32_t* out_counts) {
    if (!h || !out_tokens || !out_counts) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (!e->prefilled) return SD2_ERR_STATE;
    launch_set_flag(e->stream, e->ws.forced_on, 0);
    sd2_status st = check_launch(e, "round");
    if (st != SD2_OK) return st;
    return run_round(e, out_tokens, out_counts);
}

sd2_status sd2_round_forced(sd2_handle_t h, const int32_t* forced, int32_t* out_tokens, int32_t* out_counts) {
    if (!h || !forced || !out_tokens || !out_counts) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (!e->prefilled) return SD2_ERR_STATE;
    size_t bytes = sizeof(int32_t) * (size_t)e->batch * (e->cfg.k + 2);
    hipError_t err = hipMemcpyAsync(e->ws.forced, forced, bytes, hipMemcpyDeviceToDevice, e->stream);
    if (err != hipSuccess) return hip_fail(e, err, "hipMemcpyAsync");
    launch_set_flag(e->stream, e->ws.forced_on, 1);
    sd2_status st = check_launch(e, "round_forced");
    if (st != SD2_OK) return st;
    return run_round(e, out_tokens, out_counts);
}

sd2_status sd2_destroy(sd2_handle_t h) {
    if (!h) return SD2_OK;
    Engine* e = reinterpret_cast<Engine*>(h);
    drop_graph(*e);
    if (e->prof) {
        for (int i = 0; i < kProfMax; ++i) {
            if (e->prof[i].a) (void)hipEventDestroy(e->prof[i].a);
            if (e->prof[i].b) (void)hipEventDestroy(e->prof[i].b);
        }
        delete[] e->prof;
        e->prof = nullptr;
    }
    if (e->static_slot) {
        // the next handle on this device clears the same memory: let this one's work finish first
        (void)hipStreamSynchronize(e->stream);
        std::lock_guard<std::mutex> lock(g_static_mu);
        g_static[e->static_device].live = false;
        return SD2_OK;
    }
    delete e;
    return SD2_OK;
}

sd2_status sd2_profile(sd2_handle_t h, int32_t enable) {
    if (!h) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (enable && !e->prof) {
        // all timing events are created here, outside any stream capture
        e->prof = new (std::nothrow) ProfEntry[kProfMax]();
        if (!e->prof) return SD2_ERR_INVALID_ARG;
        for (int i = 0; i < kProfMax; ++i) {
            hipError_t err = hipEventCreateWithFlags(&e->prof[i].a, hipEventDefault);
            if (err == hipSuccess) err = hipEventCreateWithFlags(&e->prof[i].b, hipEventDefault);
            if (err != hipSuccess) return hip_fail(e, err, "hipEventCreate");
        }
    }
    if ((bool)enable != e->prof_on) {
        drop_graph(*e);  // the next round is recorded again, with or without timing events
        e->prof_on = enable != 0;
        e->prof_n = 0;
    }
    return SD2_OK;
}

sd2_status sd2_profile_read(sd2_handle_t h, int32_t cls, int32_t* launches, double* total_ms, double* bytes) {
    if (!h || !launches || !total_ms || !bytes) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    if (!e->prof_on) return SD2_ERR_STATE;
    hipError_t err = hipStreamSynchronize(e->stream);
    if (err != hipSuccess) return hip_fail(e, err, "hipStreamSynchronize");
    int n = 0;
    double ms = 0.0, by = 0.0;
    for (int i = 0; i < e->prof_n; ++i) {
        const ProfEntry& p = e->prof[i];
        if (p.cls != cls) continue;
        float t = 0.f;
        err = hipEventElapsedTime(&t, p.a, p.b);
        if (err != hipSuccess) return hip_fail(e, err, "hipEventElapsedTime");
        ++n;
        ms += t;
        by += p.bytes;
    }
    *launches = n;
    *total_ms = ms;
    *bytes = by;
    return SD2_OK;
}

sd2_status sd2_debug_read(sd2_handle_t h, int32_t what, void* dst_host, size_t bytes) {
    if (!h || !dst_host) return SD2_ERR_INVALID_ARG;
    Engine* e = reinterpret_cast<Engine*>(h);
    int B = e->batch, k = e->cfg.k, V = e->mv.dm.vocab;
    if (B < 1) return SD2_ERR_STATE;
    const void* src = nullptr;
    size_t want = 0;
    switch (what) {
        case SD2_DBG_LOGITS_V: src = e->ws.logits_v; want = sizeof(float) * (size_t)B * (k + 1) * V; break;
        case SD2_DBG_LOGITS_D: src = e->ws.logits_d; want = sizeof(float) * (size_t)B * k * V; break;
        case SD2_DBG_STEER: src = e->ws.steer; want = sizeof(float) * (size_t)B * e->md.dm.d_model; break;
        case SD2_DBG_UBIAS:
            if (!e->mlp) return SD2_ERR_STATE;
            src = e->ws.ubias;
            want = sizeof(float) * (size_t)B * e->nbias;
            break;
        case SD2_DBG_OWN_DRAFTS: src = e->ws.own_drafts; want = sizeof(int32_t) * (size_t)B * k; break;
        case SD2_DBG_OWN_N: src = e->ws.own_n; want = sizeof(int32_t) * (size_t)B; break;
        case SD2_DBG_OWN_Y: src = e->ws.own_y; want = sizeof(int32_t) * (size_t)B; break;
        case SD2_DBG_HIST: src = e->ws.hist; want = sizeof(int32_t) * (size_t)B * e->cap; break;
        case SD2_DBG_STATE: want = sizeof(int32_t) * (size_t)B * 5; break;
        case SD2_DBG_HIDDEN_V: src = e->ws.hidden_dbg; want = sizeof(float) * (size_t)B * (k + 1) * e->mv.dm.d_model; break;
        case SD2_DBG_PATH: want = sizeof(int32_t) * 2; break;
        case SD2_DBG_NONFINITE: src = e->ws.nonfinite; want = sizeof(int32_t); break;
        case SD2_DBG_TRACE:
            if (!e->mk.trace) return SD2_ERR_STATE;
            src = e->mk.trace;
            want = sizeof(int64_t) * (size_t)kMkMaxLaunch * kMkTracePhases;
            break;
        default: return SD2_ERR_INVALID_ARG;
    }
    if (bytes != want) return SD2_ERR_INVALID_ARG;
    if (what == SD2_DBG_PATH) {
        int32_t* out = (int32_t*)dst_host;
        out[0] = e->mk.active ? 1 : 0;
        out[1] = 0;
        if (e->mk.err) {
            hipError_t err = hipStreamSynchronize(e->stream);
            if (err == hipSuccess) err = hipMemcpy(&out[1], e->mk.err, sizeof(int32_t), hipMemcpyDeviceToHost);
            if (err != hipSuccess) return hip_fail(e, err, "hipMemcpy");
        }
        return SD2_OK;
    }
    if (what == SD2_DBG_HIDDEN_V) {
        launch_rmsnorm_rows(e->stream, e->mk.active ? e->mk.final_x : e->mv.x, B * (k + 1), e->mv.dm.d_model,
                            e->mv.final_norm, e->bf16, e->mv.dm.rms_eps, e->ws.hidden_dbg);
        sd2_status st = check_launch(e, "debug_read");
        if (st != SD2_OK) return st;
    }
    hipError_t err = hipStreamSynchronize(e->stream);
    if (err != hipSuccess) return hip_fail(e, err, "hipStreamSynchronize");
    if (what == SD2_DBG_STATE) {
        int32_t* out = (int32_t*)dst_host;
        const int32_t* cols[5] = {e->ws.t, e->ws.len_v, e->ws.len_d, e->ws.produced, e->ws.done};
        int32_t* tmp = new (std::nothrow) int32_t[B];
        if (!tmp) return SD2_ERR_INVALID_ARG;
        for (int c = 0; c < 5; ++c) {
            err = hipMemcpy(tmp, cols[c], sizeof(int32_t) * B, hipMemcpyDeviceToHost);
            if (err != hipSuccess) {
                delete[] tmp;
                return hip_fail(e, err, "hipMemcpy");
            }
            for (int b = 0; b < B; ++b) out[b * 5 + c] = tmp[b];
        }
        delete[] tmp;
        return SD2_OK;
    }
    err = hipMemcpy(dst_host, src, want, hipMemcpyDeviceToHost);
    if (err != hipSuccess) return hip_fail(e, err, "hipMemcpy");
    if (what == SD2_DBG_NONFINITE) {
        // the read clears the flag (outside any captured round, so a plain memset)
        err = hipMemsetAsync(e->ws.nonfinite, 0, sizeof(int32_t), e->stream);
        if (err == hipSuccess) err = hipStreamSynchronize(e->stream);
        if (err != hipSuccess) return hip_fail(e, err, "hipMemsetAsync");
    }
    return SD2_OK;
}

}  // extern "C"
