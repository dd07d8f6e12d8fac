// Persistent per-launch "round program" kernel (one cooperative launch per drafter step and one
// for the verifier's block pass): the host records the sequence of phases of a launch once, the
// kernel walks it, with a grid barrier between phases (a KV-head counter wait before attention).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sd2.h"

namespace sd2 {

constexpr int kMkWaves = 8;                      // weight-streaming waves per workgroup
constexpr int kMkThreads = kMkWaves * 64;
constexpr int kMkMaxRows = 16;                   // activation rows per launch
constexpr int kMkSpan = 64;                      // cache positions per attention unit
constexpr int kMkMaxNq = 32;                     // query vectors per (sequence, KV head): rows x query heads per KV head
constexpr int kMkMaxKR = 4096;                   // K-range staged per workgroup
constexpr int kMkLdsBudget = 150 * 1024;         // dynamic LDS per workgroup
constexpr int kMkLine = 32;                      // ints per 128-byte line
constexpr int kMkBarInts = 16 * kMkLine;         // barrier state: per XCD group a counter line (0..7) and a release line (8..15)

enum MkOp : int32_t { kMkGemv = 1, kMkAttn = 2 };
enum MkX : int32_t { kMkXBuf = 0, kMkXEmbed = 1, kMkXAttn = 2 };

// One phase.  GEMV: Y (op)= W . xn over `tiles` 16-row tiles, K cut into S ranges of KR columns;
// each unit is a tile times a 512-column slice per wave, wpu waves per tile (gate|up: a tile is
// 16 features with a gate and an up sub-tile when subs == 2, else 8 gate + 8 up rows).  ATTN:
// causal GQA attention of the launch's rows over the cache of layer `layer`, in units of
// (sequence, KV head, group of up to 8 query vectors, 64-position span).
struct MkPhase {
    int32_t op, mode, K, tiles, S, KR, wpu, subs, nseg, xsrc, res_embed, ldy;
    int32_t seg_tiles[3];
    int32_t layer, nsplit;
    int32_t defer;           // ATTN: leave the span partials unmerged (the next projection merges them)
    int32_t kvsig;           // Q|K|V: count every finished tile in on its KV head's counter
    int32_t kvwait;          // ATTN: wait for the unit's KV head counter instead of a grid barrier
    int32_t ub_ld;           // row stride of ubias (per sequence)
    const uint16_t* W[3];
    const float* X;          // activation rows [M][K] (kMkXBuf), or attention partials (kMkXAttn)
    const uint16_t* gamma;   // RMSNorm gain, or null (no norm)
    const float* xres;       // Add: residual rows [M][ldy] (unless res_embed)
    float* Y;                // output
    float* ss_out;           // Add: per-16-column sums of squares of the new residual, or null
    const int32_t* out_map;  // Store: output row of each row (-1: none), or null
    float* part;             // S > 1: [tiles][S][subs][256] partial tiles
    int32_t* cnt;            // S > 1: arrival counter per tile; ATTN: per (sequence, KV head, query group)
    float* qout;             // Qkv: queries [M][H*hd]; ATTN: query source
    float* aout;             // ATTN: output [M][H*hd]
    float* apart;            // ATTN: partials [M][H][nsplit][hd+4] (outputs, span max, span sum)
    const float* ubias;      // MLP steering, per sequence: SwiGLU, this layer's up-projection bias; Add (down
                             // projection), the bias after the MLP; or null
};

// Launch-wide arguments.
struct MkArgs {
    const MkPhase* prog;
    int32_t nphase;
    int32_t kind;            // 0: drafter step j, 1: verifier block
    int32_t j, M, rps;       // drafter step, rows, rows per sequence
    int32_t batch, k, cap, max_batch, d, H, Hkv, hd;
    float eps, scale;
    const int32_t *t, *len_d, *done, *hist, *drafts;
    const float* steer;      // [max_batch][d] (drafter launches)
    const uint16_t* embed;   // [vocab][d]
    int32_t vocab, add_steer;
    float *kc, *vc;
    const float *rcos, *rsin;
    const uint16_t* dummy;   // 1 KB of zeros (loads of absent units)
    const uint16_t* ones;    // kMkMaxKR bf16 ones (gain of projections without a norm)
    int32_t* bar;            // kMkBarInts
    uint32_t bar_gen;        // grid barriers completed on this state before this launch
    int32_t* qc;             // this model's KV-head counters (one line each): Q|K|V tiles finished
    uint32_t qc_base;        // their value before this launch
    int32_t qc_tpk;          // Q|K|V tiles per KV head (each counter grows by this per layer)
    int32_t* err;            // set to 1 if a grid barrier timed out
    int64_t* trace;          // profiling: end time of every phase (device clock, 100 MHz), or null
    int32_t G;
};

constexpr int kMkQcLines = 64;   // KV heads per model the counters cover
constexpr int kMkMaxLaunch = 33;  // drafter steps 1..k (k <= 32) and the verifier block (index 0)
constexpr int kMkTracePhases = 1024;  // phase end times kept per launch when profiling

// Engine-side state of the round-program path (device buffers live in the workspace).
struct MkState {
    MkPhase* prog;        // phase lists of all launches
    int prog_cap;         // capacity in phases
    char* arena;          // per-launch activation buffers
    size_t arena_bytes;   // its size (a recorded program must fit in it)
    int32_t* bar;         // grid-barrier state
    uint32_t bar_gen;     // grid barriers completed so far (a launch adds one per phase after the first,
                          // except attention phases that wait on KV-head counters)
    int32_t* qc;          // [2 models][kMkQcLines] KV-head counters (verifier, drafter)
    uint32_t qc_total[2]; // their current value per model
    int32_t* err;         // barrier time-out flag
    int32_t* cnt;         // hand-off counters
    uint16_t* dummy;      // 1 KB of zeros
    uint16_t* ones;       // kMkMaxKR bf16 ones
    int max_batch;        // largest supported batch (0: path unavailable)
    int batch;            // batch the lists were recorded for
    int G;                // workgroups (= compute units)
    size_t lds;           // dynamic LDS per workgroup
    int off[kMkMaxLaunch], n[kMkMaxLaunch];
    double bytes[kMkMaxLaunch];  // weight bytes streamed by each launch
    bool active;
    const float* tap_x[3]; // verifier launch: residual rows after the steering tap blocks (h, m, l)
    float* final_x;       // verifier launch: final residual rows [M][d_V]
    float* final_ss;      //   and their 16-column sums of squares
    int64_t* trace;       // [kMkMaxLaunch][kMkTracePhases] phase end times of the last profiled round
};

struct Engine;

// Host side (mk.hip).
int mk_max_batch(const sd2_config& c);                 // 0: the round-program path is unavailable
size_t mk_arena_bytes(const sd2_config& c, int batch);
int mk_phase_count(const sd2_config& c);
size_t mk_counter_ints(const sd2_config& c);
void mk_init_buffers(Engine& e);
// Records the launches' phase lists for `batch` and copies them to the device.
bool mk_build(Engine& e, int batch);
// Launches drafter step j (1..k) or the verifier block (j = 0).
hipError_t mk_launch(Engine& e, int j);

}  // namespace sd2
