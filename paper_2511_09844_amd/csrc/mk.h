// Persistent per-launch "round program" kernel: one cooperative launch per drafter step and one
// for the verifier's block pass.  The host records the phases of each launch once; the kernel
// walks them with a grid barrier between phases.
//
// A workgroup has two kinds of waves:
//   - streaming waves stream the weight units of every projection phase of the launch, in order,
//     two units in flight per wave, across phase boundaries; each unit is contracted with the
//     staged activation rows (MFMA) into a partial tile in LDS;
//   - control waves run the grid barrier, stage each projection's input rows into LDS, sum the
//     partial tiles, apply the epilogue and write every output of the phase; they also run the
//     embedding, attention and split-K hand-offs.
// Weight loads therefore never wait on barriers, stores or activation loads.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sd2.h"

namespace sd2 {

constexpr int kMkQW = 4;                         // streaming waves per workgroup
constexpr int kMkCW = 4;                         // control waves per workgroup
constexpr int kMkThreads = (kMkQW + kMkCW) * 64;
constexpr int kMkMaxRows = 16;                   // activation rows per launch
constexpr int kMkParts = 32;                     // partial-tile slots (LDS ring)
constexpr int kMkPartBytes = 1024;               // one partial tile: up to 16 x 16 floats
constexpr int kMkActBudget = 120 * 1024;         // LDS for staged activation rows (hi and lo planes)
constexpr int kMkLine = 32;                      // ints per 128-byte line
constexpr int kMkBarInts = 8 * kMkLine;          // barrier: one counter line per workgroup group

enum MkOp : int32_t { kMkEmbed = 0, kMkProj = 1, kMkAttn = 2 };

// One phase.
//   EMBED: x0 = E[tok] (+ steering) for the launch's rows, as fp32 rows, gained hi/lo rows and
//          sums of squares of 16-column slices.
//   PROJ:  Y (op)= W . xn, W row-major [N][K] bf16.  Work unit: 16 "lane rows" x 512 columns of
//          weights; a tile is h = 16 / f output features, its K range split into f interleaved
//          32-column groups (lane row j * h + i streams feature i, group j), so one load
//          instruction reads h rows x 64 f bytes.  K is cut into S ranges of KR columns (split
//          over workgroups, summed by a hand-off when S > 1); a sub-tile has KR / (512 f) units.
//   ATTN:  causal GQA attention of the launch's rows over layer `layer` of the cache; units
//          (sequence, query head, span of `span` positions), partials merged by the last span.
struct MkPhase {
    int32_t op, mode;
    int32_t K, tiles, S, KR, f, h, subs, nkc;   // projection geometry (nkc: units per sub-tile)
    int32_t seg_tiles0, seg_tiles1;              // Q|K|V: tiles of Q, of K (V follows)
    int32_t stage;                               // ordinal of this projection in the launch
    int32_t layer, nsplit, span;                 // attention; layer also for the K/V append
    int32_t ldy;                                 // row stride of Y (floats)
    int32_t nss_in, nss_out;                     // sums-of-squares slices per row: input (0: no norm), output
    int32_t nout;                                // columns of the hi/lo output rows
    int32_t pad0, pad1;
    const uint16_t* W[3];
    const uint16_t* xhl;      // input rows as bf16 hi and lo planes [2][M][K]
    const float* ss_in;       // [M][nss_in] sums of squares of the un-gained input rows
    const uint16_t* gnext;    // gain folded into the hi/lo output (the consumer's norm), or null
    const float* xres;        // Add: residual rows [M][ldy]
    float* Y;                 // fp32 output: Add: new residual; Store: logits; Q|K|V: queries; Embed: x0
    uint16_t* yhl;            // hi/lo output planes [2][M][nout], or null
    float* ss_out;            // [M][nss_out] sums of squares of the output rows (Add, Embed)
    const int32_t* out_map;   // Store: destination row per row (-1: none), or null
    float* part;              // S > 1: [tiles][S][subs][256] partial tiles
    int32_t* cnt;             // S > 1: counter per tile; ATTN: counter per (sequence, head)
    float* apart;             // ATTN: partials [M][H][nsplit][hd + 2] (output, span max, span sum)
    const float* q;           // ATTN: queries [M][H * hd]
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
    int32_t* bar;            // kMkBarInts
    uint32_t bar_base;       // barriers completed by earlier launches (counters are never reset)
    int32_t* err;            // [0]: set to 1 if a wait timed out
    int64_t* trace;          // profiling: end time of every phase (device clock, 100 MHz), or null
    int32_t G;
    int32_t act_bytes;       // LDS bytes of the staged-rows region (the partial-tile ring follows)
};

constexpr int kMkMaxLaunch = 33;  // drafter steps 1..k (k <= 32) and the verifier block (index 0)
constexpr int kMkTracePhases = 1024;  // phase end times kept per launch when profiling

// Engine-side state of the round-program path (device buffers live in the workspace).
struct MkState {
    MkPhase* prog;        // phase lists of all launches
    int prog_cap;         // capacity in phases
    char* arena;          // per-launch activation buffers
    int32_t* bar;         // grid-barrier counters
    uint32_t bar_base;    // barriers completed since the counters were cleared
    int32_t* err;         // wait time-out flag
    int32_t* cnt;         // hand-off counters (split-K tiles, attention heads)
    int max_batch;        // largest supported batch (0: path unavailable)
    int batch;            // batch the lists were recorded for
    int G;                // workgroups (= compute units)
    size_t lds;           // dynamic LDS per workgroup
    size_t act_bytes;     // of which the staged-rows region
    int off[kMkMaxLaunch], n[kMkMaxLaunch];
    double bytes[kMkMaxLaunch];  // weight bytes streamed by each launch
    bool active;
    float* final_x;       // verifier launch: final residual rows [M][d_V]
    float* final_ss;      //   and their sums of squares of final_nss slices per row
    int final_nss;
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
