// Persistent round-program kernel: one cooperative launch runs a whole drafter step (embedding
// with the steering injection, every decoder layer, the LM head) or the verifier's (k+1)-row
// block pass, as a fixed list of phases separated by grid barriers.
//
// Why: at batch 1 a decode step is a chain of ~80 dependent weight-streaming projections.  Inside
// one launch a phase boundary costs a grid barrier plus the hand-over of a few KB of activations,
// and -- the point of the wave roles below -- the weight stream does not stop there: streaming
// waves walk the weight units of all projection phases of the launch in order, with two units
// (32 KB) in flight per wave, whatever the control waves are doing.  A streaming wave only waits
// when the activation rows of a unit's phase are not staged yet or the partial-tile ring is full.
//
// Memory protocol (no device-scope fences: on this part a release fence writes back the whole
// L2): every value one workgroup produces for another is written by a control wave with
// device-scope (write-through) stores, completed (s_waitcnt) before the wave reports the phase
// done; the grid barrier follows.  Every such buffer is written once per launch before anybody
// reads it (each phase has buffers of its own; cache rows are appended before they are read), so
// no reader can hold a stale copy: caches are invalidated at launch start.
#include <hip/hip_ext.h>
#include <math.h>

#include <algorithm>
#include <vector>

#include "device_common.h"
#include "engine.h"
#include "mk.h"

namespace sd2 {

typedef __bf16 mk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mk_f4 __attribute__((ext_vector_type(4)));
typedef float mk_f2 __attribute__((ext_vector_type(2)));
typedef unsigned int mk_u4 __attribute__((ext_vector_type(4)));
// Global-address-space pointers: loads through generic pointers are "flat" and are also counted
// by the LDS counter, which would make every LDS wait a wait on memory.
typedef const __attribute__((address_space(1))) mk_u4* mk_gu4p;
typedef const __attribute__((address_space(1))) mk_f4* mk_gf4p;
typedef const __attribute__((address_space(1))) mk_f2* mk_gf2p;
typedef const __attribute__((address_space(1))) float* mk_gfp;
typedef const __attribute__((address_space(1))) int32_t* mk_gip;
typedef const __attribute__((address_space(1))) uint16_t* mk_ghp;
typedef __attribute__((address_space(1))) void* mk_gvp;
typedef __attribute__((address_space(3))) void* mk_lvp;
// Phase descriptors are read through the constant address space: uniform reads become scalar
// loads, which a streaming wave does not have to wait for behind its weight loads.
typedef const __attribute__((address_space(4))) MkPhase* mk_cph;
__device__ __forceinline__ mk_cph mk_phase(const MkArgs& a, int p) { return (mk_cph)(a.prog + p); }

constexpr int kQW = kMkQW;
constexpr int kCW = kMkCW;
constexpr int kP = kMkParts;
constexpr long kMkTimeout = 50000000;  // 0.5 s of the 100 MHz device clock per wait

__device__ __forceinline__ int mk_ld(int32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ int mk_add(int32_t* p, int v) { return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void mk_sti(int32_t* p, int v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void mk_stf(float* p, float v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void mk_stu(uint16_t* p, uint32_t v) {
    __hip_atomic_store((uint32_t*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float mk_ldg(const float* p) { return *(mk_gfp)p; }
__device__ __forceinline__ float4 mk_ldg4(const float* p) {
    mk_f4 v = *(mk_gf4p)p;
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float2 mk_ldg2(const float* p) {
    mk_f2 v = *(mk_gf2p)p;
    return make_float2(v.x, v.y);
}
__device__ __forceinline__ float mk_ldbf(const uint16_t* p) { return bf16_to_f32(*(mk_ghp)p); }
__device__ __forceinline__ int mk_ldi(const int32_t* p) { return *(mk_gip)p; }
__device__ __forceinline__ void mk_vmwait() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
__device__ __forceinline__ void mk_lgkmwait() { __builtin_amdgcn_s_waitcnt(0xC07F); } // lgkmcnt(0)

// bf16 hi/lo split of x: hi = rne(x), lo = rne(x - hi); returned as two bf16 bit patterns.
__device__ __forceinline__ uint32_t mk_hilo(float x) {
    const __bf16 h = (__bf16)x;
    const __bf16 l = (__bf16)(x - (float)h);
    return (uint32_t)__builtin_bit_cast(uint16_t, h) | ((uint32_t)__builtin_bit_cast(uint16_t, l) << 16);
}

// Workgroup-local control state.
struct MkCtl {
    int act_cnt;             // staging completions: kCW per projection phase
    int done_cnt;            // phase completions: kCW per phase
    int open;                // last phase whose grid barrier has opened
    int abort;               // a wait timed out: every wave leaves
    int att;                 // attention: control-wave arrivals (kCW per shared unit)
    int pflag[kP];           // unit whose partial tile the slot holds (-1: none)
    int pfree[kP];           // first unit allowed to write the slot
    float rms[kMkMaxRows];
};

// The control block and the row plan are reached through LDS-typed references: a generic
// (flat) access would also count as a memory access, and a streaming wave waiting for it would
// wait for its weight loads.
typedef __attribute__((address_space(3))) MkCtl MkCtlL;
typedef int __attribute__((address_space(3))) lds_int;
__device__ __forceinline__ int lds_get(const lds_int& v) { return *(const volatile lds_int*)&v; }
__device__ __forceinline__ void lds_put(lds_int& v, int x) { *(volatile lds_int*)&v = x; }

// Poll `ready` with a bounded wait.  Returns false when this wave must leave (time-out here, or
// another wave of the workgroup timed out); a time-out also sets the launch's error flag.
template <typename F>
__device__ __forceinline__ bool mk_wait(MkCtlL& ctl, const MkArgs& a, F&& ready) {
    if (ready()) return true;
    const long t0 = (long)wall_clock64();
    while (true) {
        __builtin_amdgcn_s_sleep(1);
        if (ready()) return true;
        if (lds_get(ctl.abort)) return false;
        if ((long)wall_clock64() - t0 > kMkTimeout) {
            lds_put(ctl.abort, 1);
            mk_sti(a.err, 1);
            return false;
        }
    }
}

// Row plan of the launch, one entry per activation row (position -1: inactive row).
struct MkRows {
    int pos[kMkMaxRows], seq[kMkMaxRows], tok[kMkMaxRows];
};
typedef __attribute__((address_space(3))) MkRows MkRowsL;

__device__ __forceinline__ void mk_plan(const MkArgs& a, MkRowsL& rp) {
    const int r = threadIdx.x;
    if (r >= kMkMaxRows) return;
    int b = 0, pos = -1, tok = 0;
    if (r < a.M) {
        if (a.kind == 1) {
            b = r / (a.k + 1);
            const int i = r % (a.k + 1);
            if (b < a.batch && !a.done[b]) {
                const int t = a.t[b];
                pos = t - 1 + i;
                tok = i == 0 ? a.hist[(size_t)b * a.cap + t - 1] : a.drafts[b * a.k + i - 1];
            }
        } else if (a.j == 1) {
            b = r >> 1;
            const int i = r & 1;
            if (b < a.batch && !a.done[b]) {
                const int t = a.t[b], m = t - a.len_d[b];
                if (i == 1) pos = t - 1;
                else if (m == 2) pos = t - 2;
                if (pos >= 0) tok = a.hist[(size_t)b * a.cap + pos];
            }
        } else {
            b = r;
            if (b < a.batch && !a.done[b]) {
                pos = a.t[b] + a.j - 2;
                tok = a.drafts[b * a.k + a.j - 2];
            }
        }
    }
    rp.pos[r] = pos;
    rp.seq[r] = b < a.max_batch ? b : 0;
    rp.tok[r] = tok < 0 ? 0 : (tok >= a.vocab ? a.vocab - 1 : tok);
}

// Units of a projection phase owned by this workgroup (0 for other phases).
__device__ __forceinline__ int mk_units_of(mk_cph ph, int G) {
    if (ph->op != kMkProj) return 0;
    const int S = ph->S, gs = G / S, gt = (int)blockIdx.x / S;
    const int nt = ph->tiles > gt ? (ph->tiles - gt + gs - 1) / gs : 0;
    return nt * ph->subs * ph->nkc;
}

// Cursor over the launch's unit sequence: phase p holds units [base, base + n) of this workgroup.
struct MkCur {
    int p, base, n;
};
__device__ __forceinline__ void mk_seek(const MkArgs& a, MkCur& c, int gu) {
    while (c.p < a.nphase && gu >= c.base + c.n) {
        c.base += c.n;
        ++c.p;
        c.n = c.p < a.nphase ? mk_units_of(mk_phase(a, c.p), a.G) : 0;
    }
}

// ---------------------------------------------------------------------------------------------
// Streaming waves.
// ---------------------------------------------------------------------------------------------
// Address of this lane's first weight element of unit `uu` of phase `ph`: lane row l = lane & 15
// is feature i = l % h of the tile, column group j = l / h; lane quarter q = lane >> 4 takes 8
// columns.  Q|K|V tiles pair rotate-half partners: the first h/2 rows of a tile are dims
// (h/2) jj + i of a head, the other h/2 rows the same dims + hd/2.
__device__ __forceinline__ const uint16_t* mk_unit_ptr(const MkArgs& a, mk_cph ph, int uu, int lane) {
    const int nkc = ph->nkc, subs = ph->subs, S = ph->S, h = ph->h, K = ph->K;
    const int c = uu % nkc, ts = uu / nkc, sub = ts % subs, t = ts / subs;
    const int s = (int)blockIdx.x % S, gt = (int)blockIdx.x / S, gs = a.G / S;
    const int tile = gt + t * gs;
    const int l = lane & 15, q = lane >> 4, j = l / h, i = l % h;
    const uint16_t* base;
    size_t row;
    if (ph->mode == kEpiQkv) {
        int seg = 0, lt = tile;
        if (lt >= ph->seg_tiles0) {
            lt -= ph->seg_tiles0;
            seg = 1;
            if (lt >= ph->seg_tiles1) {
                lt -= ph->seg_tiles1;
                seg = 2;
            }
        }
        const int per_head = a.hd / h, hh = lt / per_head, jj = lt % per_head, half = h / 2;
        const int ii = half * jj + (i % half);
        row = (size_t)hh * a.hd + (i < half ? ii : a.hd / 2 + ii);
        base = ph->W[seg];
    } else {
        row = (size_t)tile * h + i;
        base = ph->W[ph->mode == kEpiSwiglu ? sub : 0];
    }
    return base + row * K + (size_t)s * ph->KR + (size_t)c * 512 * ph->f + 32 * j + 8 * q;
}

template <int F>
__device__ __forceinline__ void mk_issue_f(mk_u4 (&b)[16], const uint16_t* p) {
    mk_gu4p g = (mk_gu4p)p;
#pragma unroll
    for (int st = 0; st < 16; ++st) b[st] = __builtin_nontemporal_load(g + st * 4 * F);
}
// Issue a unit's 16 loads.  Past the last unit of the launch the same 16 loads read the phase
// list instead (valid memory; the data is never used): every path then has the same number of
// loads in flight, so the compiler's wait counts stay those of two full buffers.
__device__ __forceinline__ void mk_issue(mk_u4 (&b)[16], const MkArgs& a, const MkCur& c, int gu, int lane) {
    const uint16_t* p = (const uint16_t*)a.prog + 8 * lane;
    int f = 1;
    if (c.p < a.nphase) {
        const mk_cph ph = mk_phase(a, c.p);
        p = mk_unit_ptr(a, ph, gu - c.base, lane);
        f = ph->f;
    }
    if (f == 4) mk_issue_f<4>(b, p);
    else if (f == 2) mk_issue_f<2>(b, p);
    else mk_issue_f<1>(b, p);
}

// Contract a weight unit (A operand, lane row x 8 columns per step) with the staged rows (B
// operand: column n = j * (16/F) + m reads row m of the hi or lo plane at column group j), then
// fold the F column groups: the result for (feature i, row m) ends in lane m + 16 (i >> 2),
// element i & 3, and goes to the partial slot as [m][i].
template <int F>
__device__ __forceinline__ void mk_mma_put(const mk_u4 (&b)[16], const uint16_t* act, int ldk, int M, int cc, int lane,
                                           float* slot) {
    constexpr int MP = 16 / F, H = 16 / F;
    const int n = lane & 15, q = lane >> 4, jj = n / MP, m = n % MP;
    const int mr = m < M ? m : M - 1;  // columns of absent rows repeat a real row (results unused)
    const uint16_t* ph = act + (size_t)mr * ldk + cc * 512 * F + 32 * jj + 8 * q;
    const uint16_t* pl = ph + (size_t)M * ldk;
    mk_f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 16; ++st) {
        if ((st & 3) == 0) asm volatile("" ::: "memory");  // at most four steps of LDS reads in flight
        const mk_u4 xh = *(const mk_u4*)(ph + 32 * F * st);
        const mk_u4 xl = *(const mk_u4*)(pl + 32 * F * st);
        const mk_bf16x8 w = __builtin_bit_cast(mk_bf16x8, b[st]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, __builtin_bit_cast(mk_bf16x8, xh), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, __builtin_bit_cast(mk_bf16x8, xl), acc, 0, 0, 0);
    }
    // group j of (feature i, row m) sits 80 j / F lanes further; sum the unmodified values
    mk_f4 sum = acc;
#pragma unroll
    for (int j = 1; j < F; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum[r] += __shfl(acc[r], (lane + j * 80 / F) & 63, 64);
    const int g = lane >> 4, mm = lane & 15;
    if (mm < MP && g < H / 4) *(mk_f4*)(slot + mm * H + 4 * g) = sum;
}

__device__ __forceinline__ bool mk_compute(const mk_u4 (&b)[16], const MkArgs& a, MkCtlL& ctl, const MkCur& c, int gu,
                                           int lane, char* smem) {
    const mk_cph ph = mk_phase(a, c.p);
    const int stage = ph->stage, f = ph->f, ldk = ph->KR + 8, nkc = ph->nkc;
    const int cc = (gu - c.base) % nkc;
    if (!mk_wait(ctl, a, [&] { return lds_get(ctl.act_cnt) >= kCW * (stage + 1); })) return false;
    const int slot = gu % kP;
    if (!mk_wait(ctl, a, [&] { return lds_get(ctl.pfree[slot]) >= gu; })) return false;
    const uint16_t* act = (const uint16_t*)smem;
    float* ps = (float*)(smem + a.act_bytes) + slot * 256;
    if (f == 4) mk_mma_put<4>(b, act, ldk, a.M, cc, lane, ps);
    else if (f == 2) mk_mma_put<2>(b, act, ldk, a.M, cc, lane, ps);
    else mk_mma_put<1>(b, act, ldk, a.M, cc, lane, ps);
    mk_lgkmwait();
    if (lane == 0) lds_put(ctl.pflag[slot], gu);
    return true;
}

__device__ __forceinline__ void mk_stream(const MkArgs& a, MkCtlL& ctl, char* smem, int wave, int lane) {
    // units wave, wave + kQW, wave + 2 kQW, ... of the launch, two in flight
    MkCur c0{0, 0, mk_units_of(mk_phase(a, 0), a.G)};
    MkCur c1 = c0;
    int gu0 = wave, gu1 = wave + kQW;
    mk_seek(a, c0, gu0);
    mk_seek(a, c1, gu1);
    mk_u4 b0[16], b1[16];
    mk_issue(b0, a, c0, gu0, lane);
    mk_issue(b1, a, c1, gu1, lane);
    while (c0.p < a.nphase) {
        if (!mk_compute(b0, a, ctl, c0, gu0, lane, smem)) return;
        gu0 += 2 * kQW;
        mk_seek(a, c0, gu0);
        mk_issue(b0, a, c0, gu0, lane);
        if (c1.p >= a.nphase) break;
        if (!mk_compute(b1, a, ctl, c1, gu1, lane, smem)) return;
        gu1 += 2 * kQW;
        mk_seek(a, c1, gu1);
        mk_issue(b1, a, c1, gu1, lane);
    }
}

// ---------------------------------------------------------------------------------------------
// Control waves.
// ---------------------------------------------------------------------------------------------
// Grid barrier opening phase p (p >= 1).  Control wave 0 waits until every control wave of the
// workgroup has finished phase p-1 (stores completed), counts the workgroup in on its group's
// counter, then polls all eight group counters.  Counters only grow: barrier b of the process
// is complete when every group counter has reached b times its workgroup count.
__device__ __forceinline__ bool mk_open(const MkArgs& a, MkCtlL& ctl, int p, int cw, int lane) {
    if (cw != 0) return mk_wait(ctl, a, [&] { return lds_get(ctl.open) >= p; });
    if (!mk_wait(ctl, a, [&] { return lds_get(ctl.done_cnt) >= kCW * p; })) return false;
    const unsigned per = (unsigned)a.G / 8u;
    const unsigned target = (a.bar_base + (unsigned)p) * per;
    if (lane == 0) mk_add(a.bar + ((int)blockIdx.x & 7) * kMkLine, 1);
    const long t0 = (long)wall_clock64();
    while (true) {
        bool ok = true;
        if (lane < 8) ok = (int)((unsigned)mk_ld(a.bar + lane * kMkLine) - target) >= 0;
        if (__ballot(!ok) == 0) break;
        __builtin_amdgcn_s_sleep(1);
        if (lds_get(ctl.abort)) return false;
        if ((long)wall_clock64() - t0 > kMkTimeout) {
            lds_put(ctl.abort, 1);
            mk_sti(a.err, 1);
            return false;
        }
    }
    if (lane == 0) lds_put(ctl.open, p);
    return true;
}

// Stage this workgroup's K range of the phase's input rows (hi and lo planes) into LDS with
// direct-to-LDS loads (1 KB per instruction), and, for a normed input, 1/rms of every row from
// the producer's sums of squares (control wave cw takes rows cw, cw + kCW, ...; its sums are
// requested before its share of the rows, so one wait covers both).  The staging counter (kCW
// per projection) covers rows and 1/rms.
__device__ __forceinline__ bool mk_stage(const MkArgs& a, MkCtlL& ctl, mk_cph ph, char* smem, int cw, int lane) {
    const int M = a.M, KR = ph->KR, K = ph->K, ldk = KR + 8;
    const int s = (int)blockIdx.x % ph->S;
    const int per = KR / 512, nblk = 2 * M * per;
    const int nss = ph->nss_in;
    const float* ssp = ph->ss_in;
    constexpr int RPW = kMkMaxRows / kCW;  // rows per control wave
    float sm[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        sm[r] = 0.f;
        const int m = cw + kCW * r;
        if (m < M)
            for (int t0 = 0; t0 < nss; t0 += 1024)
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int t = t0 + 64 * u + lane;
                    if (t < nss) sm[r] += mk_ldg(ssp + (size_t)m * nss + t);
                }
    }
    uint16_t* act = (uint16_t*)smem;
    for (int b = cw; b < nblk; b += kCW) {
        const int row = b / per, cb = b % per;
        const uint16_t* src = ph->xhl + (size_t)row * K + (size_t)s * KR + cb * 512 + 8 * lane;
        uint16_t* dst = act + (size_t)row * ldk + cb * 512;
        __builtin_amdgcn_global_load_lds((mk_gvp)(void*)src, (mk_lvp)(void*)dst, 16, 0, 0);
    }
    mk_vmwait();
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const int m = cw + kCW * r;
        const float v = wave_sum(sm[r]);
        if (lane == 0 && m < M) ctl.rms[m] = nss > 0 ? rsqrtf(v / (float)K + a.eps) : 1.0f;
    }
    mk_lgkmwait();
    if (lane == 0) __hip_atomic_fetch_add((int*)&ctl.act_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int stage = ph->stage;
    return mk_wait(ctl, a, [&] { return lds_get(ctl.act_cnt) >= kCW * (stage + 1); });
}

// Hi/lo planes of one output value per lane, stored in pairs of columns: the lane with the even
// column writes both (its neighbour lane holds the odd column).
__device__ __forceinline__ void mk_put_hl(uint16_t* yhl, int M, int nout, int m, int col, float x, bool valid) {
    const uint32_t v = mk_hilo(x);
    const uint32_t nb = (uint32_t)__shfl((int)v, ((int)threadIdx.x + 1) & 63, 64);
    if (valid && (col & 1) == 0) {
        mk_stu(yhl + (size_t)m * nout + col, (v & 0xffffu) | (nb << 16));
        mk_stu(yhl + ((size_t)M + m) * nout + col, (v >> 16) | (nb & 0xffff0000u));
    }
}

// Q|K|V output (feature i of tile `tile`): segment (0 Q, 1 K, 2 V), head, dim, and the RoPE
// frequency index of the rotate-half pair.
struct MkQkv {
    int seg, hh, dim, ii;
};
__device__ __forceinline__ MkQkv mk_qkv_of(const MkArgs& a, mk_cph ph, int tile, int i) {
    const int h = ph->h, half = h / 2;
    int seg = 0, lt = tile;
    if (lt >= ph->seg_tiles0) {
        lt -= ph->seg_tiles0;
        seg = 1;
        if (lt >= ph->seg_tiles1) {
            lt -= ph->seg_tiles1;
            seg = 2;
        }
    }
    const int per_head = a.hd / h, hh = lt / per_head, jj = lt % per_head;
    const int ii = half * jj + (i % half);
    return MkQkv{seg, hh, i < half ? ii : a.hd / 2 + ii, ii};
}

// Epilogue inputs of output o of a tile, requested before the tile's partial sums are waited
// for: Add: residual and the next norm's gain; Q|K|V: RoPE cos and sin; Store: output row.
__device__ __forceinline__ void mk_epi_pre(const MkArgs& a, const MkRowsL& rp, mk_cph ph, int tile, int o, float& e0,
                                           float& e1, int& ei) {
    const int h = ph->h, m = o / h, i = o % h;
    const bool valid = m < a.M;
    const int mode = ph->mode;
    e0 = 0.f;
    e1 = 1.f;
    ei = m;
    if (!valid) return;
    if (mode == kEpiStore) {
        if (ph->out_map) ei = mk_ldi(ph->out_map + m);
    } else if (mode == kEpiAdd) {
        const int col = tile * h + i;
        e0 = mk_ldg(ph->xres + (size_t)m * ph->ldy + col);
        if (ph->gnext) e1 = mk_ldbf(ph->gnext + col);
    } else if (mode == kEpiQkv) {
        const MkQkv g = mk_qkv_of(a, ph, tile, i);
        if (g.seg < 2) {
            const int pos = rp.pos[m], pp = pos < 0 ? 0 : pos;
            e0 = mk_ldg(a.rcos + (size_t)pp * (a.hd / 2) + g.ii);
            e1 = mk_ldg(a.rsin + (size_t)pp * (a.hd / 2) + g.ii);
        }
    }
}

// Epilogue of one output per lane: (feature i, row m) of tile `tile`, value v0 (v1: the up half
// of a SwiGLU pair), prefetched inputs e0, e1, ei.  All 64 lanes call it (shuffles).
__device__ __forceinline__ void mk_epi(const MkArgs& a, const MkRowsL& rp, mk_cph ph, int tile, int o, float v0,
                                       float v1, float e0, float e1, int ei) {
    const int h = ph->h, M = a.M;
    const int m = o / h, i = o % h;
    const bool valid = m < M;  // M <= h, so o < h * h
    const int mode = ph->mode;
    if (mode == kEpiStore) {
        const int col = tile * h + i;
        if (valid && ei >= 0) mk_stf(ph->Y + (size_t)ei * ph->ldy + col, v0);
    } else if (mode == kEpiAdd) {
        const int col = tile * h + i;
        const float nv = valid ? e0 + v0 : 0.f;
        if (valid) mk_stf(ph->Y + (size_t)m * ph->ldy + col, nv);
        mk_put_hl(ph->yhl, M, ph->nout, m, col, e1 * nv, valid);
        float sq = nv * nv;
        for (int off = 1; off < h; off <<= 1) sq += __shfl_xor(sq, off, 64);
        if (valid && i == 0) mk_stf(ph->ss_out + (size_t)m * ph->nss_out + tile, sq);
    } else if (mode == kEpiSwiglu) {
        const int col = tile * h + i;
        const float out = valid ? silu(v0) * v1 : 0.f;
        mk_put_hl(ph->yhl, M, ph->nout, m, col, out, valid);
    } else {  // Q|K|V: rotate-half RoPE on Q and K, cache append of K and V
        const int half = h / 2;
        const float partner = __shfl_xor(v0, half, 64);
        if (!valid) return;
        const MkQkv g = mk_qkv_of(a, ph, tile, i);
        const int pos = rp.pos[m];
        float out = v0;
        if (g.seg < 2) out = i < half ? v0 * e0 - partner * e1 : v0 * e0 + partner * e1;
        if (g.seg == 0) {
            mk_stf(ph->Y + (size_t)m * a.H * a.hd + g.hh * a.hd + g.dim, out);
        } else if (pos >= 0) {
            const size_t idx =
                ((((size_t)ph->layer * a.max_batch + rp.seq[m]) * a.Hkv + g.hh) * a.cap + pos) * a.hd + g.dim;
            mk_stf(g.seg == 1 ? a.kc + idx : a.vc + idx, out);
        }
    }
}

// Sum the partial tiles of this workgroup's tiles (tile t goes to control wave t % kCW), scale by
// 1/rms, and finish each tile: epilogue, or the split-K hand-off.
__device__ __forceinline__ bool mk_finish(const MkArgs& a, MkCtlL& ctl, const MkRowsL& rp, mk_cph ph, char* smem,
                                          int cw, int lane, int base) {
    const int S = ph->S, gs = a.G / S, gt = (int)blockIdx.x / S, s = (int)blockIdx.x % S;
    const int nt = ph->tiles > gt ? (ph->tiles - gt + gs - 1) / gs : 0;
    const int subs = ph->subs, nkc = ph->nkc, h = ph->h;
    const int nout = h * h;  // partial-tile entries [m][i], m < 16 / f = h
    const float* parts = (const float*)(smem + a.act_bytes);
    for (int t = cw; t < nt; t += kCW) {
        const int tile = gt + t * gs;
        float e0[4], e1[4];
        int ei[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (64 * k < nout) mk_epi_pre(a, rp, ph, tile, lane + 64 * k, e0[k], e1[k], ei[k]);
        float v0[4] = {0.f, 0.f, 0.f, 0.f}, v1[4] = {0.f, 0.f, 0.f, 0.f};
        for (int sub = 0; sub < subs; ++sub)
            for (int cc = 0; cc < nkc; ++cc) {
                const int gu = base + (t * subs + sub) * nkc + cc, slot = gu % kP;
                if (!mk_wait(ctl, a, [&] { return lds_get(ctl.pflag[slot]) == gu; })) return false;
                const float* ps = parts + slot * 256;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int o = lane + 64 * k;
                    if (o < nout) {
                        if (sub == 0) v0[k] += ps[o];
                        else v1[k] += ps[o];
                    }
                }
                mk_lgkmwait();
                if (lane == 0) lds_put(ctl.pfree[slot], gu + kP);
            }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int o = lane + 64 * k, m = o / h;
            const float r = m < a.M ? ctl.rms[m] : 0.f;
            v0[k] *= r;
            v1[k] *= r;
        }
        if (S > 1) {
            float* pt = ph->part + ((size_t)tile * S + s) * subs * 256;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int o = lane + 64 * k;
                if (o < nout) {
                    mk_stf(pt + o, v0[k]);
                    if (subs == 2) mk_stf(pt + 256 + o, v1[k]);
                }
            }
            mk_vmwait();
            int last = 0;
            if (lane == 0) {
                const int prev = mk_add(ph->cnt + tile, 1);
                last = prev == S - 1;
                if (last) mk_sti(ph->cnt + tile, 0);
            }
            last = __shfl(last, 0, 64);
            if (!last) continue;
            const float* p0 = ph->part + (size_t)tile * S * subs * 256;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v0[k] = 0.f;
                v1[k] = 0.f;
            }
            for (int s0 = 0; s0 < S; ++s0)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int o = lane + 64 * k;
                    if (o < nout) {
                        v0[k] += mk_ldg(p0 + (size_t)s0 * subs * 256 + o);
                        if (subs == 2) v1[k] += mk_ldg(p0 + (size_t)s0 * subs * 256 + 256 + o);
                    }
                }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (64 * k < nout) mk_epi(a, rp, ph, tile, lane + 64 * k, v0[k], v1[k], e0[k], e1[k], ei[k]);
    }
    return true;
}

// Embedding rows (+ steering for drafter launches): x0 fp32, gained hi/lo rows, sums of squares
// of 16-column slices.  Slice gg of all rows goes to one control wave.
__device__ __forceinline__ void mk_embed(const MkArgs& a, const MkRowsL& rp, mk_cph ph, int cw, int lane) {
    const int d = a.d, M = a.M, ng = d / 16;
    for (int gg = (int)blockIdx.x + a.G * cw; gg < ng; gg += a.G * kCW) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int o = lane + 64 * k, m = o / 16, c = o % 16;
            const bool valid = m < M;
            const int col = gg * 16 + c;
            float x = 0.f;
            if (valid && rp.pos[m] >= 0) {
                x = mk_ldbf(a.embed + (size_t)rp.tok[m] * d + col);
                if (a.add_steer) x += mk_ldg(a.steer + (size_t)rp.seq[m] * d + col);
            }
            if (valid) mk_stf(ph->Y + (size_t)m * d + col, x);
            const float g = (valid && ph->gnext) ? mk_ldbf(ph->gnext + col) : 1.0f;
            mk_put_hl(ph->yhl, M, d, m, col, g * x, valid);
            float sq = x * x;
            for (int off = 1; off < 16; off <<= 1) sq += __shfl_xor(sq, off, 64);
            if (valid && c == 0) mk_stf(ph->ss_out + (size_t)m * ng + gg, sq);
        }
    }
}

// Attention geometry for head dim HD: lanes per scored position, sub-span per control wave
// (positions), head dims per lane when scoring, position groups and head dims per lane when
// forming outputs.  A unit (sequence, query head, span of kCW sub-spans) is shared by the kCW
// control waves of a workgroup.
template <int HD>
struct MkAttnGeo {
    static constexpr int LPP = HD >= 128 ? HD / 64 : 1;
    static constexpr int SP = 64 / LPP;
    static constexpr int DPL = HD / LPP;
    static constexpr int PS = HD >= 64 ? 1 : 64 / HD;
    static constexpr int DV = HD >= 64 ? HD / 64 : 1;
    static constexpr int PPL = SP / PS;
    static constexpr int USP = kCW * SP;
};

// Attention.  Each control wave scores its sub-span of the unit (lane pair / lane = position)
// against the sequence's query rows, forms un-normalised outputs (lane = head-dim columns) and
// leaves (output, max, sum) per row in LDS; after the control waves meet, control wave 0 merges
// the sub-spans, then either writes the normalised output (the only live span) or stores the
// unit's partial, and the last unit of a (sequence, head) to arrive merges all live units in
// span order.  Outputs are written as hi/lo planes (the O projection's input).
template <int HD>
__device__ __forceinline__ bool mk_attn(const MkArgs& a, MkCtlL& ctl, const MkRowsL& rp, mk_cph ph, char* smem,
                                        int cw, int lane, int& gen) {
    using Gm = MkAttnGeo<HD>;
    constexpr int LPP = Gm::LPP, SP = Gm::SP, DPL = Gm::DPL, PS = Gm::PS, DV = Gm::DV, PPL = Gm::PPL, USP = Gm::USP;
    constexpr int SUB = kMkMaxRows * (HD + 2);  // one sub-span partial: [row][HD outputs, max, sum]
    const int M = a.M, rps = a.rps, H = a.H, Gq = a.H / a.Hkv;
    const int nsplit = ph->nsplit, nseq = M / rps;
    const int nunit = nseq * H * nsplit;
    float* qs = (float*)smem + cw * (kMkMaxRows * HD + SP);  // [rps][HD] pre-scaled queries
    float* pr = qs + kMkMaxRows * HD;                       // [SP] probabilities of the current row
    float* subs = (float*)smem + kCW * (kMkMaxRows * HD + SP);  // [2][kCW][SUB]
    uint16_t* out = ph->yhl;
    const int ldo = H * HD;
    for (int u = (int)blockIdx.x; u < nunit; u += a.G) {
        const int sp = u % nsplit, hh = (u / nsplit) % H, sq = u / (nsplit * H);
        const int kvh = hh / Gq, r0 = sq * rps;
        int maxq = -1;
        for (int i = 0; i < rps; ++i) maxq = max(maxq, rp.pos[r0 + i]);
        const int p0 = sp * USP;
        const int nl = maxq >= 0 ? min(nsplit, maxq / USP + 1) : 0;
        if (nl == 0) {
            if (sp == 0 && cw == 0)
                for (int e = lane; e < rps * HD; e += 64)
                    mk_put_hl(out, M, ldo, r0 + e / HD, hh * HD + e % HD, 0.f, true);
            continue;
        }
        if (maxq < p0) continue;  // dead unit: no work and no hand-off
        const int pw = p0 + cw * SP;
        const int nvalid = maxq >= pw ? min(SP, maxq - pw + 1) : 0;
        float* sb = subs + ((gen & 1) * kCW + cw) * SUB;
        if (nvalid > 0) {
            const size_t head_base = (((size_t)ph->layer * a.max_batch + rp.seq[r0]) * a.Hkv + kvh) * a.cap * HD;
            const float* kg = a.kc + head_base + (size_t)pw * HD;
            const float* vg = a.vc + head_base + (size_t)pw * HD;
            // all loads of the sub-span first: this lane's K slice, its V columns, the query rows
            const int pos = lane / LPP, part = lane % LPP;
            float4 kr[DPL / 4];
            {
                const int jr = pos < nvalid ? pos : nvalid - 1;
#pragma unroll
                for (int t = 0; t < DPL / 4; ++t) kr[t] = mk_ldg4(kg + (size_t)jr * HD + part * DPL + 4 * t);
            }
            const int pgrp = lane / (64 / PS), dcol = (lane % (64 / PS)) * DV;
            float vv[PPL][DV];
#pragma unroll
            for (int j = 0; j < PPL; ++j) {
                const int pj = pgrp * PPL + j;
                const int jr = pj < nvalid ? pj : nvalid - 1;
                if (DV == 2) {
                    const float2 v2 = mk_ldg2(vg + (size_t)jr * HD + dcol);
                    vv[j][0] = v2.x;
                    vv[j][DV - 1] = v2.y;
                } else {
                    vv[j][0] = mk_ldg(vg + (size_t)jr * HD + dcol);
                }
            }
            for (int e = lane * 4; e < rps * HD; e += 256) {
                const int i = e / HD, dd = e % HD;
                const float4 v = mk_ldg4(ph->q + (size_t)(r0 + i) * H * HD + hh * HD + dd);
                *(float4*)(qs + i * HD + dd) = make_float4(v.x * a.scale, v.y * a.scale, v.z * a.scale, v.w * a.scale);
            }
            for (int i = 0; i < rps; ++i) {
                const float4* qr = (const float4*)(qs + i * HD + part * DPL);
                float sc = 0.f;
#pragma unroll
                for (int t = 0; t < DPL / 4; ++t) {
                    const float4 qv = qr[t], kv = kr[t];
                    sc += qv.x * kv.x + qv.y * kv.y + qv.z * kv.z + qv.w * kv.w;
                }
                if (LPP == 2) sc += __shfl_xor(sc, 1, 64);
                const int qp = rp.pos[r0 + i];
                const float v = (pos < nvalid && pw + pos <= qp) ? sc : -INFINITY;
                const float mx = wave_max(v);
                const float ev = v == -INFINITY ? 0.f : expf(v - mx);
                const float sm = wave_sum(part == 0 ? ev : 0.f);
                if (part == 0) pr[pos] = ev;
                float o[DV];
#pragma unroll
                for (int dv = 0; dv < DV; ++dv) o[dv] = 0.f;
                const float* pp = pr + pgrp * PPL;
#pragma unroll
                for (int jj = 0; jj < PPL; ++jj) {
                    const float pj = pp[jj];
#pragma unroll
                    for (int dv = 0; dv < DV; ++dv) o[dv] += pj * vv[jj][dv];
                }
                if (PS > 1)
#pragma unroll
                    for (int dv = 0; dv < DV; ++dv) o[dv] += __shfl_xor(o[dv], 32, 64);
                float* sr = sb + i * (HD + 2);
                if (pgrp == 0)
#pragma unroll
                    for (int dv = 0; dv < DV; ++dv) sr[dcol + dv] = o[dv];
                if (lane == 0) {
                    sr[HD] = mx;
                    sr[HD + 1] = sm;
                }
            }
        } else if (lane < rps) {
            sb[lane * (HD + 2) + HD] = -INFINITY;
            sb[lane * (HD + 2) + HD + 1] = 0.f;
        }
        // the control waves meet; control wave 0 merges the sub-spans
        mk_lgkmwait();
        ++gen;
        if (lane == 0) __hip_atomic_fetch_add((int*)&ctl.att, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (!mk_wait(ctl, a, [&] { return lds_get(ctl.att) >= kCW * gen; })) return false;
        if (cw != 0) continue;
        const float* sb0 = subs + ((gen - 1) & 1) * kCW * SUB;
        float* pa0 = ph->apart + (((size_t)r0 * H + hh) * nsplit + sp) * (HD + 2);
        for (int e = lane; e < rps * HD; e += 64) {
            const int i = e / HD, dd = e % HD;
            float mw[kCW], Mx = -INFINITY;
#pragma unroll
            for (int w = 0; w < kCW; ++w) {
                mw[w] = sb0[w * SUB + i * (HD + 2) + HD];
                Mx = fmaxf(Mx, mw[w]);
            }
            float L = 0.f, O = 0.f;
            if (Mx != -INFINITY)
#pragma unroll
                for (int w = 0; w < kCW; ++w)
                    if (mw[w] != -INFINITY) {
                        const float wt = expf(mw[w] - Mx);
                        L += wt * sb0[w * SUB + i * (HD + 2) + HD + 1];
                        O += wt * sb0[w * SUB + i * (HD + 2) + dd];
                    }
            if (nl == 1) {
                mk_put_hl(out, M, ldo, r0 + i, hh * HD + dd, L > 0.f ? O / L : 0.f, true);
            } else {
                float* pa = pa0 + (size_t)i * H * nsplit * (HD + 2);
                mk_stf(pa + dd, O);
                if (dd == 0) {
                    mk_stf(pa + HD, Mx);
                    mk_stf(pa + HD + 1, L);
                }
            }
        }
        if (nl == 1) continue;
        mk_vmwait();
        int last = 0;
        if (lane == 0) {
            int32_t* c = ph->cnt + sq * H + hh;
            const int prev = mk_add(c, 1);
            last = prev == nl - 1;
            if (last) mk_sti(c, 0);
        }
        last = __shfl(last, 0, 64);
        if (!last) continue;
        // merge the nl live units: lane -> (query row, 4 head dims); row max and normaliser from
        // every unit's (max, sum), sixteen units per round trip
        constexpr int D4 = HD / 4;
        for (int e = lane; e < rps * D4; e += 64) {
            const int i = e / D4, dd = (e % D4) * 4;
            float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
            if (rp.pos[r0 + i] >= 0) {
                const float* pb = ph->apart + ((size_t)(r0 + i) * H + hh) * nsplit * (HD + 2);
                float Mx = -INFINITY, L = 0.f;
                float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int s0 = 0; s0 < nl; s0 += 16) {
                    float4 v[16];
                    float2 ml[16];
#pragma unroll
                    for (int t = 0; t < 16; ++t) {
                        const float* e2 = pb + (size_t)min(s0 + t, nl - 1) * (HD + 2);
                        v[t] = mk_ldg4(e2 + dd);
                        ml[t] = mk_ldg2(e2 + HD);
                    }
                    float cm = -INFINITY;
#pragma unroll
                    for (int t = 0; t < 16; ++t)
                        if (s0 + t < nl) cm = fmaxf(cm, ml[t].x);
                    if (cm == -INFINITY) continue;
                    if (cm > Mx) {
                        const float scl = Mx == -INFINITY ? 0.f : expf(Mx - cm);
                        L *= scl;
                        O.x *= scl;
                        O.y *= scl;
                        O.z *= scl;
                        O.w *= scl;
                        Mx = cm;
                    }
#pragma unroll
                    for (int t = 0; t < 16; ++t) {
                        if (s0 + t >= nl || ml[t].x == -INFINITY) continue;
                        const float w = expf(ml[t].x - Mx);
                        L += w * ml[t].y;
                        O.x += w * v[t].x;
                        O.y += w * v[t].y;
                        O.z += w * v[t].z;
                        O.w += w * v[t].w;
                    }
                }
                if (L > 0.f) {
                    const float inv = 1.f / L;
                    r = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
                }
            }
            const uint32_t x0 = mk_hilo(r.x), x1 = mk_hilo(r.y), x2 = mk_hilo(r.z), x3 = mk_hilo(r.w);
            uint16_t* ob = out + (size_t)(r0 + i) * ldo + hh * HD + dd;
            mk_stu(ob, (x0 & 0xffffu) | (x1 << 16));
            mk_stu(ob + 2, (x2 & 0xffffu) | (x3 << 16));
            mk_stu(ob + (size_t)M * ldo, (x0 >> 16) | (x1 & 0xffff0000u));
            mk_stu(ob + (size_t)M * ldo + 2, (x2 >> 16) | (x3 & 0xffff0000u));
        }
    }
    return true;
}

__device__ __forceinline__ void mk_control(const MkArgs& a, MkCtlL& ctl, const MkRowsL& rp, char* smem, int cw, int lane) {
    int base = 0, gen = 0;
    if (a.trace && blockIdx.x == 0 && cw == 0 && lane == 0) a.trace[0] = wall_clock64();
    for (int p = 0; p < a.nphase; ++p) {
        const mk_cph ph = mk_phase(a, p);
        if (p > 0 && !mk_open(a, ctl, p, cw, lane)) return;
        const int op = ph->op;
        bool ok = true;
        if (op == kMkProj) {
            ok = mk_stage(a, ctl, ph, smem, cw, lane) && mk_finish(a, ctl, rp, ph, smem, cw, lane, base);
            base += mk_units_of(ph, a.G);
        } else if (op == kMkAttn) {
            if (a.hd == 128) ok = mk_attn<128>(a, ctl, rp, ph, smem, cw, lane, gen);
            else if (a.hd == 64) ok = mk_attn<64>(a, ctl, rp, ph, smem, cw, lane, gen);
            else ok = mk_attn<32>(a, ctl, rp, ph, smem, cw, lane, gen);
        } else {
            mk_embed(a, rp, ph, cw, lane);
        }
        if (!ok) return;
        mk_vmwait();  // this wave's stores of the phase are complete
        if (lane == 0) __hip_atomic_fetch_add((int*)&ctl.done_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (a.trace && blockIdx.x == 0 && cw == 0 && lane == 0 && p + 1 < kMkTracePhases) a.trace[p + 1] = wall_clock64();
    }
}

__global__ __launch_bounds__(kMkThreads) void k_mk(MkArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ MkRows rp_;
    __shared__ MkCtl ctl_;
    MkRowsL& rp = *(MkRowsL*)&rp_;
    MkCtlL& ctl = *(MkCtlL*)&ctl_;
    const int tid = threadIdx.x;
    mk_plan(a, rp);
    if (tid < kP) {
        ctl.pflag[tid] = -1;
        ctl.pfree[tid] = tid;
    }
    if (tid == 0) {
        ctl.act_cnt = 0;
        ctl.done_cnt = 0;
        ctl.open = 0;
        ctl.abort = 0;
        ctl.att = 0;
    }
    __syncthreads();
    // the wave index is uniform within a wave; saying so keeps every value derived from it
    // (unit ids, phase cursors, descriptor addresses) in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    if (wave < kQW) mk_stream(a, ctl, smem, wave, lane);
    else mk_control(a, ctl, rp, smem, wave - kQW, lane);
}

// =============================================================================================
// Host side: phase lists.
// =============================================================================================
namespace {

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

struct Arena {
    char* base;
    size_t off;
    template <typename T>
    T* take(size_t n) {
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += up256(n * sizeof(T));
        return p;
    }
};

// Geometry of a projection of M rows, N outputs, contraction K: the widest column-group fold f
// (f = 4, 2, 1: tiles of 16 / f features, so one load instruction reads 16 / f rows) whose B
// columns hold the rows (M <= 16 / f), then the fewest K ranges S whose staged rows fit in LDS.
struct MkGeo {
    int f, h, S, KR, nkc;
    size_t act;
};
MkGeo mk_geo(int M, int N, int K, int G, int hd, bool qkv) {
    MkGeo best{0, 0, 0, 0, 0, 0};
    for (int f = 4; f >= 1; f /= 2) {
        const int h = 16 / f;
        if (M > 16 / f || N % h) continue;
        if (qkv && (hd % h)) continue;
        for (int S = 1; S <= 8; S *= 2) {
            if (K % S || (G > 0 && G % S)) continue;
            const int KR = K / S;
            if (KR % (512 * f)) continue;
            const size_t act = (size_t)2 * M * (KR + 8) * 2;
            if (act > (size_t)kMkActBudget) continue;
            return MkGeo{f, h, S, KR, KR / (512 * f), act};
        }
    }
    return best;
}

int mk_span(int hd) {  // positions per attention unit: kCW sub-spans
    return hd == 128 ? MkAttnGeo<128>::USP : hd == 64 ? MkAttnGeo<64>::USP : MkAttnGeo<32>::USP;
}
int mk_nsplit(int cap, int hd) { return (cap + mk_span(hd) - 1) / mk_span(hd); }
size_t mk_attn_lds(int hd) {
    const int sp = mk_span(hd) / kCW;
    return (size_t)kCW * ((size_t)kMkMaxRows * hd + sp) * 4 + (size_t)2 * kCW * kMkMaxRows * (hd + 2) * 4;
}

// Phases of one launch of model m with M rows (rps per sequence); appends to `out` when given.
// Returns false when a shape is not supported.  `act` receives the largest LDS region needed.
struct MkRec {
    size_t act = 0;
    double bytes = 0.0;
    float* final_x = nullptr;
    float* final_ss = nullptr;
    int final_nss = 0;
};
bool mk_record(const sd2_config& c, const ModelDev& m, bool verifier, int M, int rps, int j, int G, Arena& ar,
               const Workspace* ws, std::vector<MkPhase>* out, int32_t* cnt, MkRec& rec) {
    const sd2_dims& d = m.dm;
    const int hd = d.d_model / d.n_heads;
    const int L = d.n_layers, H = d.n_heads, Hkv = d.n_kv_heads, F = d.d_ff, dm = d.d_model;
    if (M > kMkMaxRows || M < 1 || rps < 1 || M % rps) return false;
    if (hd != 32 && hd != 64 && hd != 128) return false;
    if (dm % 16) return false;
    const int nsplit = mk_nsplit(c.max_seq_len, hd);
    rec.act = std::max(rec.act, mk_attn_lds(hd));
    const size_t cnt_tiles = (size_t)std::max(std::max(d.vocab, F), dm) / 4 + 1;
    int stage = 0;
    auto proj = [&](int mode, int N, int K, int subs, MkPhase& ph) -> bool {
        MkGeo g = mk_geo(M, N, K, G, hd, mode == kEpiQkv);
        if (!g.f) return false;
        ph.op = kMkProj;
        ph.mode = mode;
        ph.K = K;
        ph.tiles = N / g.h;
        ph.S = g.S;
        ph.KR = g.KR;
        ph.f = g.f;
        ph.h = g.h;
        ph.subs = subs;
        ph.nkc = g.nkc;
        ph.stage = stage++;
        ph.cnt = cnt;
        if (g.S > 1) ph.part = ar.take<float>((size_t)ph.tiles * g.S * subs * 256);
        rec.act = std::max(rec.act, g.act);
        rec.bytes += (double)N * K * 2.0 * subs;
        return ph.tiles <= (int)cnt_tiles;
    };
    const void* const* W = m.layer;
    // embedding phase: x0 rows, hi/lo with the first layer's attention-norm gain, 16-column sums
    MkPhase em{};
    em.op = kMkEmbed;
    float* x_prev = ar.take<float>((size_t)M * dm);
    uint16_t* xhl_prev = ar.take<uint16_t>((size_t)2 * M * dm);
    float* ss_prev = ar.take<float>((size_t)M * (dm / 16));
    int nss_prev = dm / 16;
    em.Y = x_prev;
    em.yhl = xhl_prev;
    em.ss_out = ss_prev;
    em.nss_out = nss_prev;
    em.gnext = (const uint16_t*)W[kAttnNorm];
    if (out) out->push_back(em);
    for (int l = 0; l < L; ++l) {
        const void* const* Wl = W + (size_t)l * 9;
        const void* gnext = l + 1 < L ? W[(size_t)(l + 1) * 9 + kAttnNorm] : m.final_norm;
        float* q = ar.take<float>((size_t)M * H * hd);
        uint16_t* att = ar.take<uint16_t>((size_t)2 * M * H * hd);
        float* apart = ar.take<float>((size_t)M * H * nsplit * (hd + 2));
        float* xa = ar.take<float>((size_t)M * dm);
        uint16_t* xahl = ar.take<uint16_t>((size_t)2 * M * dm);
        uint16_t* hhl = ar.take<uint16_t>((size_t)2 * M * F);
        float* xf = ar.take<float>((size_t)M * dm);
        uint16_t* xfhl = ar.take<uint16_t>((size_t)2 * M * dm);
        MkPhase qkv{};
        if (!proj(kEpiQkv, (H + 2 * Hkv) * hd, dm, 1, qkv)) return false;
        qkv.nss_in = nss_prev;
        qkv.ss_in = ss_prev;
        qkv.xhl = xhl_prev;
        qkv.W[0] = (const uint16_t*)Wl[kWq];
        qkv.W[1] = (const uint16_t*)Wl[kWk];
        qkv.W[2] = (const uint16_t*)Wl[kWv];
        qkv.seg_tiles0 = H * hd / qkv.h;
        qkv.seg_tiles1 = Hkv * hd / qkv.h;
        qkv.Y = q;
        qkv.layer = l;
        MkPhase at{};
        at.op = kMkAttn;
        at.layer = l;
        at.nsplit = nsplit;
        at.span = mk_span(hd);
        at.q = q;
        at.yhl = att;
        at.nout = H * hd;
        at.apart = apart;
        at.cnt = cnt + cnt_tiles;
        MkPhase o{};
        if (!proj(kEpiAdd, dm, H * hd, 1, o)) return false;
        o.xhl = att;
        o.W[0] = (const uint16_t*)Wl[kWo];
        o.xres = x_prev;
        o.Y = xa;
        o.ldy = dm;
        o.yhl = xahl;
        o.nout = dm;
        o.gnext = (const uint16_t*)Wl[kFfnNorm];
        o.nss_out = o.tiles;
        o.ss_out = ar.take<float>((size_t)M * o.tiles);
        MkPhase gu{};
        if (!proj(kEpiSwiglu, F, dm, 2, gu)) return false;
        gu.xhl = xahl;
        gu.nss_in = o.nss_out;
        gu.ss_in = o.ss_out;
        gu.W[0] = (const uint16_t*)Wl[kWg];
        gu.W[1] = (const uint16_t*)Wl[kWu];
        gu.yhl = hhl;
        gu.nout = F;
        MkPhase dn{};
        if (!proj(kEpiAdd, dm, F, 1, dn)) return false;
        dn.xhl = hhl;
        dn.W[0] = (const uint16_t*)Wl[kWd];
        dn.xres = xa;
        dn.Y = xf;
        dn.ldy = dm;
        dn.yhl = xfhl;
        dn.nout = dm;
        dn.gnext = (const uint16_t*)gnext;
        dn.nss_out = dn.tiles;
        dn.ss_out = ar.take<float>((size_t)M * dn.tiles);
        if (out) {
            out->push_back(qkv);
            out->push_back(at);
            out->push_back(o);
            out->push_back(gu);
            out->push_back(dn);
        }
        x_prev = xf;
        xhl_prev = xfhl;
        ss_prev = dn.ss_out;
        nss_prev = dn.nss_out;
    }
    rec.final_x = x_prev;
    rec.final_ss = ss_prev;
    rec.final_nss = nss_prev;
    MkPhase lm{};
    if (!proj(kEpiStore, d.vocab, dm, 1, lm)) return false;
    lm.xhl = xhl_prev;
    lm.nss_in = nss_prev;
    lm.ss_in = ss_prev;
    lm.W[0] = (const uint16_t*)m.lm_head;
    lm.ldy = d.vocab;
    if (ws) {
        lm.Y = verifier ? ws->logits_v : ws->logits_d;
        lm.out_map = verifier ? nullptr : ws->lm_map_d + (size_t)(j - 1) * 2 * c.max_batch;
    }
    if (out) out->push_back(lm);
    return true;
}

size_t mk_lds_total(size_t act) { return up256(act) + (size_t)kP * kMkPartBytes; }

}  // namespace

// Largest batch for which both launch kinds are supported (0: none).
int mk_max_batch(const sd2_config& c) {
    if (c.dtype != SD2_BF16) return 0;
    ModelDev mv{}, md{};
    mv.dm = c.verifier;
    md.dm = c.drafter;
    for (int b = std::min(c.max_batch, kMkMaxRows); b >= 1; --b) {
        Arena ar{nullptr, 0};
        MkRec r1, r2, r3;
        if (mk_record(c, md, false, 2 * b, 2, 1, 0, ar, nullptr, nullptr, nullptr, r1) &&
            mk_record(c, md, false, b, 1, 2, 0, ar, nullptr, nullptr, nullptr, r2) &&
            mk_record(c, mv, true, b * (c.k + 1), c.k + 1, 0, 0, ar, nullptr, nullptr, nullptr, r3) &&
            mk_lds_total(std::max(std::max(r1.act, r2.act), r3.act)) <= 156 * 1024)
            return b;
    }
    return 0;
}

size_t mk_arena_bytes(const sd2_config& c, int batch) {
    if (batch < 1) return 0;
    ModelDev mv{}, md{};
    mv.dm = c.verifier;
    md.dm = c.drafter;
    size_t mx = 0;
    {
        Arena ar{nullptr, 0};
        MkRec r;
        mk_record(c, md, false, 2 * batch, 2, 1, 0, ar, nullptr, nullptr, nullptr, r);
        mx = std::max(mx, ar.off);
    }
    {
        Arena ar{nullptr, 0};
        MkRec r;
        mk_record(c, mv, true, batch * (c.k + 1), c.k + 1, 0, 0, ar, nullptr, nullptr, nullptr, r);
        mx = std::max(mx, ar.off);
    }
    return mx;
}

int mk_phase_count(const sd2_config& c) {
    return c.k * (5 * c.drafter.n_layers + 2) + 5 * c.verifier.n_layers + 2;
}

size_t mk_counter_ints(const sd2_config& c) {
    const int n = std::max(std::max(c.verifier.vocab, c.drafter.vocab),
                           std::max(std::max(c.verifier.d_ff, c.drafter.d_ff), std::max(c.verifier.d_model, c.drafter.d_model)));
    return (size_t)n / 4 + 1 + (size_t)kMkMaxRows * std::max(c.verifier.n_heads, c.drafter.n_heads) + 64;
}

void mk_init_buffers(Engine& e) {
    MkState& s = e.mk;
    if (!s.prog) return;
    (void)hipMemsetAsync(s.cnt, 0, sizeof(int32_t) * mk_counter_ints(e.cfg), e.stream);
    (void)hipMemsetAsync(s.bar, 0, sizeof(int32_t) * kMkBarInts, e.stream);
    (void)hipMemsetAsync(s.err, 0, sizeof(int32_t) * 64, e.stream);
    s.bar_base = 0;
}

bool mk_build(Engine& e, int batch) {
    MkState& s = e.mk;
    s.active = false;
    if (!s.prog || batch > s.max_batch || batch < 1 || getenv("SD2_NO_MK")) return false;
    if (e.cfg.k + 1 > kMkMaxLaunch) return false;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    int cus = 0, coop = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop) return false;
    if (cus < 8 || cus % 8) return false;  // eight workgroup groups of equal size (barrier counters)
    s.G = cus;
    std::vector<MkPhase> prog;
    size_t act = 0;
    const sd2_config& c = e.cfg;
    for (int j = 1; j <= c.k; ++j) {
        Arena ar{s.arena, 0};
        MkRec r;
        s.off[j] = (int)prog.size();
        if (!mk_record(c, e.md, false, j == 1 ? 2 * batch : batch, j == 1 ? 2 : 1, j, s.G, ar, &e.ws, &prog, s.cnt, r))
            return false;
        s.n[j] = (int)prog.size() - s.off[j];
        s.bytes[j] = r.bytes;
        act = std::max(act, r.act);
    }
    {
        Arena ar{s.arena, 0};
        MkRec r;
        s.off[0] = (int)prog.size();
        if (!mk_record(c, e.mv, true, batch * (c.k + 1), c.k + 1, 0, s.G, ar, &e.ws, &prog, s.cnt, r)) return false;
        s.n[0] = (int)prog.size() - s.off[0];
        s.bytes[0] = r.bytes;
        s.final_x = r.final_x;
        s.final_ss = r.final_ss;
        s.final_nss = r.final_nss;
        act = std::max(act, r.act);
    }
    if ((int)prog.size() > s.prog_cap) return false;
    s.act_bytes = up256(act);
    s.lds = mk_lds_total(act);
    if (hipFuncSetAttribute((const void*)k_mk, hipFuncAttributeMaxDynamicSharedMemorySize, (int)s.lds) != hipSuccess)
        return false;
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)k_mk, kMkThreads, s.lds) != hipSuccess || occ < 1)
        return false;
    if (hipMemcpyAsync(s.prog, prog.data(), sizeof(MkPhase) * prog.size(), hipMemcpyHostToDevice, e.stream) !=
        hipSuccess)
        return false;
    mk_init_buffers(e);
    if (hipStreamSynchronize(e.stream) != hipSuccess) return false;
    s.batch = batch;
    s.active = true;
    return true;
}

hipError_t mk_launch(Engine& e, int j) {
    MkState& s = e.mk;
    const sd2_config& c = e.cfg;
    const bool ver = j == 0;
    ModelDev& m = ver ? e.mv : e.md;
    MkArgs a{};
    a.prog = s.prog + s.off[j];
    a.nphase = s.n[j];
    a.kind = ver ? 1 : 0;
    a.j = j;
    a.M = ver ? s.batch * (c.k + 1) : (j == 1 ? 2 * s.batch : s.batch);
    a.rps = ver ? c.k + 1 : (j == 1 ? 2 : 1);
    a.batch = e.batch;
    a.k = c.k;
    a.cap = e.cap;
    a.max_batch = c.max_batch;
    a.d = m.dm.d_model;
    a.H = m.dm.n_heads;
    a.Hkv = m.dm.n_kv_heads;
    a.hd = m.hd;
    a.eps = m.dm.rms_eps;
    a.scale = 1.0f / sqrtf((float)m.hd);
    a.t = e.ws.t;
    a.len_d = e.ws.len_d;
    a.done = e.ws.done;
    a.hist = e.ws.hist;
    a.drafts = e.ws.drafts;
    a.steer = e.ws.steer;
    a.embed = (const uint16_t*)m.embed;
    a.vocab = m.dm.vocab;
    a.add_steer = ver ? 0 : 1;
    a.kc = m.kc;
    a.vc = m.vc;
    a.rcos = m.rope_cos;
    a.rsin = m.rope_sin;
    a.bar = s.bar;
    a.bar_base = s.bar_base;
    a.err = s.err;
    a.trace = (e.prof_on && s.trace) ? s.trace + (size_t)j * kMkTracePhases : nullptr;
    a.G = s.G;
    a.act_bytes = (int32_t)s.act_bytes;
    void* args[] = {&a};
    ProfEntry* pe = prof_slot(&e, kProfProgram, s.bytes[j]);
    if (pe) (void)hipEventRecord(pe->a, e.stream);
    hipError_t err = hipLaunchCooperativeKernel((const void*)k_mk, dim3(s.G), dim3(kMkThreads), args, s.lds, e.stream);
    if (pe) {
        (void)hipEventRecord(pe->b, e.stream);
        prof_commit(&e);
    }
    if (err == hipSuccess) s.bar_base += (uint32_t)(s.n[j] - 1);
    return err;
}

}  // namespace sd2
