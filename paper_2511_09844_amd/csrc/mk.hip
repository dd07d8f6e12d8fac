// Persistent round-program kernel: one cooperative launch runs a whole drafter step (embedding
// with the steering injection, every decoder layer, the LM head) or the verifier's (k+1)-row
// block pass, as a fixed list of phases.
//
// Why: a decode step at batch 1 is a chain of ~80 dependent weight-streaming projections and
// attention passes.  As separate kernels each pays the launch's own start/finish cost (several
// microseconds on this part) plus a cold start of its loads; inside one persistent launch a
// phase boundary is a grid barrier (one atomic, one store and one poll round trip after the last
// arrival) or, before attention, a wait on the counter of the unit's KV head; descriptors are
// prefetched, and the first weight unit of a projection streams while its workgroup waits.
//
// Workgroups: one per compute unit, 8 waves, every wave streaming weights.
//
// Memory protocol (no device-scope fences: on this part a release fence writes back the whole
// L2): every value one workgroup produces for another is written with device-scope
// (write-through) stores and completed (s_waitcnt) before the producer counts in at a barrier
// or on a hand-off counter; consumers read it with ordinary loads.  That is safe because every
// such buffer is written once per launch before anybody reads it (activations, residuals,
// partials each get their own region per phase; cache rows are appended before they are read,
// and a cache line holds one row), so no workgroup can hold a stale copy in its caches, which
// are invalidated at launch start.
#include <hip/hip_ext.h>
#include <math.h>

#include <algorithm>
#include <vector>

#include "device_common.h"
#include "engine.h"
#include "mk.h"

namespace sd2 {

typedef __bf16 mk_bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 mk_bf16x2 __attribute__((ext_vector_type(2)));
typedef float mk_f4 __attribute__((ext_vector_type(4)));
typedef float mk_f2 __attribute__((ext_vector_type(2)));
typedef unsigned int mk_u4 __attribute__((ext_vector_type(4)));
typedef unsigned int mk_u2 __attribute__((ext_vector_type(2)));
// Global-address-space pointers: loads through generic pointers are "flat" and are also counted
// by the LDS counter, which would make every LDS wait a wait on memory.
typedef const __attribute__((address_space(1))) mk_u4* mk_gu4p;
typedef const __attribute__((address_space(1))) mk_u2* mk_gu2p;
typedef const __attribute__((address_space(1))) mk_f4* mk_gf4p;
typedef const __attribute__((address_space(1))) mk_f2* mk_gf2p;
typedef const __attribute__((address_space(1))) float* mk_gfp;
typedef const __attribute__((address_space(1))) int32_t* mk_gip;

constexpr int kNW = kMkWaves;
constexpr int kMkPreSteps = 8;      // 64-column slices of a phase's first unit requested during its barrier
constexpr int kMkMinWG = 256;       // workgroups assumed by the LDS plans (one per compute unit)
constexpr int kNT = kMkWaves * 64;  // streaming threads
constexpr int kCtl = 0;             // thread that runs the grid barrier (no loads in flight there)
constexpr long kMkSpin = 1L << 22;  // grid-barrier polls before a workgroup gives up (reports err)

// Device-scope accesses through global-address-space pointers: through generic pointers they
// become flat instructions, and a later LDS access then waits until every earlier flat store has
// completed (a flat address might have been LDS).
typedef __attribute__((address_space(1))) int32_t* mk_gip_w;
typedef __attribute__((address_space(1))) float* mk_gfp_w;
__device__ __forceinline__ int mk_ld(int32_t* p) { return __hip_atomic_load((mk_gip_w)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ int mk_add(int32_t* p, int v) {
    return __hip_atomic_fetch_add((mk_gip_w)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void mk_sti(int32_t* p, int v) { __hip_atomic_store((mk_gip_w)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void mk_stf(float* p, float v) { __hip_atomic_store((mk_gfp_w)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ float mk_ldg(const float* p) { return *(mk_gfp)p; }
__device__ __forceinline__ float4 mk_ldg4(const float* p) {
    mk_f4 v = *(mk_gf4p)p;
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float2 mk_ldg2(const float* p) {
    mk_f2 v = *(mk_gf2p)p;
    return make_float2(v.x, v.y);
}
__device__ __forceinline__ float mk_ldbf(const uint16_t* p) {
    return bf16_to_f32(*(const __attribute__((address_space(1))) uint16_t*)p);
}
__device__ __forceinline__ int mk_ldi(const int32_t* p) { return *(mk_gip)p; }
__device__ __forceinline__ uint32_t mk_ldu(const void* p) { return *(const __attribute__((address_space(1))) uint32_t*)p; }
__device__ __forceinline__ void mk_vmwait() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Thread index seen through an empty asm: index arithmetic of a phase then stays inside that
// phase instead of being hoisted out of the phase loop, where the values of every phase kind
// would stay live together and spill.
__device__ __forceinline__ int mk_tid() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Uniform copy of a value every lane holds identically (descriptor fields read from LDS): kept in
// scalar registers instead of a stack copy of the whole descriptor.
template <typename T>
__device__ __forceinline__ T mk_uni(const T& v) {
    static_assert(sizeof(T) % 4 == 0, "32-bit words");
    uint32_t w[sizeof(T) / 4];
    __builtin_memcpy(w, &v, sizeof(T));
#pragma unroll
    for (int i = 0; i < (int)(sizeof(T) / 4); ++i) w[i] = __builtin_amdgcn_readfirstlane(w[i]);
    T r;
    __builtin_memcpy(&r, w, sizeof(T));
    return r;
}

// Wave-wide max / sum through DPP row operations (no LDS round trips): pairs, quads, half rows
// and rows by swaps and mirrors, then rows 0-3 folded into row 3 by the row broadcasts; the
// result of lane 63 is returned to every lane.
template <int CTRL, int ROWS>
__device__ __forceinline__ float mk_dpp(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v),
                                                                 CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float mk_wmax(float v) {
    v = fmaxf(v, mk_dpp<0xB1, 0xf>(v, v));   // quad_perm [1,0,3,2]
    v = fmaxf(v, mk_dpp<0x4E, 0xf>(v, v));   // quad_perm [2,3,0,1]
    v = fmaxf(v, mk_dpp<0x141, 0xf>(v, v));  // row_half_mirror
    v = fmaxf(v, mk_dpp<0x140, 0xf>(v, v));  // row_mirror
    v = fmaxf(v, mk_dpp<0x142, 0xa>(v, v));  // row_bcast:15 into rows 1 and 3
    v = fmaxf(v, mk_dpp<0x143, 0xc>(v, v));  // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float mk_wsum(float v) {
    v += mk_dpp<0xB1, 0xf>(0.f, v);
    v += mk_dpp<0x4E, 0xf>(0.f, v);
    v += mk_dpp<0x141, 0xf>(0.f, v);
    v += mk_dpp<0x140, 0xf>(0.f, v);
    v += mk_dpp<0x142, 0xa>(0.f, v);
    v += mk_dpp<0x143, 0xc>(0.f, v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Row plan of the launch, one entry per activation row (position -1: inactive row).
struct MkRows {
    int pos[kMkMaxRows], seq[kMkMaxRows], tok[kMkMaxRows];
};

__device__ __forceinline__ void mk_plan(const MkArgs& a, MkRows& rp) {
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

// ---------------------------------------------------------------------------------------------
// Projection phase.
// ---------------------------------------------------------------------------------------------
struct MkBuf {
    mk_u4 w[8][2];  // one weight unit per wave: 16 rows x 512 columns, MFMA B-operand layout
};

// Weight row streamed by lane row n of tile `tile` (Q|K|V tiles pair rotate-half partners
// i and i + hd/2, 8 of each).
struct MkW {
    const uint16_t *w0, *w1, *w2;
    int K, mode, nseg, st0, st1;
};
__device__ __forceinline__ const uint16_t* mk_row(const MkW& o, int hd, int tile, int sub, int n) {
    // gate|up: with two sub-tiles, sub 0 streams 16 gate rows and sub 1 the 16 up rows of the same
    // features; with one, lane rows 0-7 are gate rows and 8-15 the up rows of the same 8 features
    if (o.mode == kEpiSwiglu) {
        if (o.nseg == 2) return (sub ? o.w1 : o.w0) + (size_t)(tile * 16 + n) * o.K;
        return (n < 8 ? o.w0 : o.w1) + (size_t)(tile * 8 + (n & 7)) * o.K;
    }
    int seg = 0, lt = tile;
    if (o.nseg > 1 && lt >= o.st0) { lt -= o.st0; seg = 1; }
    if (o.nseg > 2 && seg == 1 && lt >= o.st1) { lt -= o.st1; seg = 2; }
    int wrow = lt * 16 + n;
    if (o.mode == kEpiQkv) {
        const int per_head = hd / 16;
        const int h = lt / per_head, jj = lt % per_head;
        wrow = h * hd + (n < 8 ? 8 * jj + n : hd / 2 + 8 * jj + (n - 8));
    }
    const uint16_t* base = seg == 0 ? o.w0 : (seg == 1 ? o.w1 : o.w2);
    return base + (size_t)wrow * o.K;
}

__device__ __forceinline__ int mk_units(int tiles, int S, int subs, int G) {
    const int gs = G / S, g = blockIdx.x / S;
    const int nt = tiles > g ? (tiles - g + gs - 1) / gs : 0;
    return nt * subs;
}

// stride 8 (16-byte words per 64 columns) for a real unit; 0 re-reads one word (absent unit)
template <int ST0 = 0, int ST1 = 8>
__device__ __forceinline__ void mk_issue(MkBuf& b, const uint16_t* wp, int stride) {
    mk_gu4p p = (mk_gu4p)wp;
#pragma unroll
    for (int st = ST0; st < ST1; ++st) {
        b.w[st][0] = p[st * stride];
        b.w[st][1] = p[st * stride + (stride >> 3)];
    }
}

// Geometry of a projection phase for this workgroup and wave, from its descriptor in LDS.
struct MkGeo {
    MkW ow;
    int s, g, gs, k0, nsub, wpu, groups, gr, kw0, subs;
    bool streams;
};
__device__ __forceinline__ MkGeo mk_geo(const MkArgs& a, const MkPhase& od, int wave) {
    MkGeo q;
    q.ow.w0 = mk_uni(od.W[0]);
    q.ow.w1 = mk_uni(od.W[1]);
    q.ow.w2 = mk_uni(od.W[2]);
    q.ow.K = mk_uni(od.K);
    q.ow.mode = mk_uni(od.mode);
    q.ow.nseg = mk_uni(od.nseg);
    q.ow.st0 = mk_uni(od.seg_tiles[0]);
    q.ow.st1 = mk_uni(od.seg_tiles[1]);
    const int tiles = mk_uni(od.tiles), S = mk_uni(od.S), KR = mk_uni(od.KR);
    q.wpu = mk_uni(od.wpu);
    q.subs = mk_uni(od.subs);
    q.s = blockIdx.x % S;
    q.g = blockIdx.x / S;
    q.gs = a.G / S;
    q.k0 = q.s * KR;
    q.nsub = mk_units(tiles, S, q.subs, a.G);
    q.groups = kNW / q.wpu;
    q.gr = wave / q.wpu;
    q.streams = wave < kNW && q.gr < q.groups;
    q.kw0 = (wave % q.wpu) * 512;
    return q;
}

// Weight unit of round r for this wave: its address for lane (n, qq), and the stride to pass to
// mk_issue (0 when the wave has no unit in that round: one word of the zero page is re-read).
__device__ __forceinline__ const uint16_t* mk_uptr(const MkArgs& a, const MkGeo& q, int r, int n, int qq, int lane,
                                                   int& stride) {
    const int u = r * q.groups + q.gr;
    if (!(q.streams && u < q.nsub)) {
        stride = 0;
        return a.dummy + lane * 8;
    }
    stride = 8;
    const int tile = q.g + (q.subs == 2 ? (u >> 1) : u) * q.gs;
    return mk_row(q.ow, a.hd, tile, q.subs == 2 ? (u & 1) : 0, n) + q.k0 + q.kw0 + 16 * qq;
}

// Fold a batch of up to 16 span partials (output, max, sum; the first cnt of them are live) into
// a running (max, sum, output) without branches, so that every load of the batch is issued before
// the first is used (a skip on "no live span" let the compiler sink the output loads behind it).
// Scaling by exp(0) = 1 and adding zero weights leave the sums exactly as with skips.
__device__ __forceinline__ void mk_fold16(const float4 (&v)[16], const float2 (&ml)[16], int cnt, float& Mx, float& L,
                                          float4& O) {
    float cm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) cm = i < cnt ? fmaxf(cm, ml[i].x) : cm;
    const float nm = fmaxf(Mx, cm);
    const float sc = Mx == -INFINITY ? 0.f : expf(Mx - nm);
    L *= sc;
    O.x *= sc;
    O.y *= sc;
    O.z *= sc;
    O.w *= sc;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const bool live = i < cnt && ml[i].x != -INFINITY;
        const float w = live ? expf(ml[i].x - nm) : 0.f;
        L += w * ml[i].y;
        O.x += w * v[i].x;
        O.y += w * v[i].y;
        O.z += w * v[i].z;
        O.w += w * v[i].w;
    }
    Mx = nm;
}

// Activation rows m0 .. m0 + R - 1 (rows past M re-read row M - 1), NJ float4 columns per thread
// (columns past the K range re-read its last one), all loads issued before any is used.
template <int R, int NJ>
__device__ __forceinline__ void mk_xload(float4 (&xv)[8][2], const float* X, int m0, int M, int K, int k0, int n4, int tid) {
#pragma unroll
    for (int mm = 0; mm < R; ++mm)
#pragma unroll
        for (int jc = 0; jc < NJ; ++jc) {
            const int m = min(m0 + mm, M - 1), c = min(tid + 512 * jc, n4 - 1);
            xv[mm][jc] = mk_ldg4(X + (size_t)m * K + k0 + 4 * c);
        }
}

// Embedding row value of activation row m, column c (+ steering for drafter launches).
__device__ __forceinline__ float mk_embed_at(const MkArgs& a, const MkRows& rp, int m, int c) {
    if (rp.pos[m] < 0) return 0.f;
    float v = mk_ldbf(a.embed + (size_t)rp.tok[m] * a.d + c);
    if (a.add_steer) v += mk_ldg(a.steer + (size_t)rp.seq[m] * a.d + c);
    return v;
}

template <bool UB>
__device__ __forceinline__ void mk_gemv(const MkArgs& a, const MkPhase& od, const MkRows& rp, char* smem, float* inv_rms,
                        int* flags, int* last_flag, MkBuf& bf) {
    // descriptor fields (od lives in LDS), uniform
    const int tid = mk_tid(), lane = tid & 63, wave = tid >> 6;
    const MkGeo q0 = mk_geo(a, od, wave);
    const MkW& ow = q0.ow;
    const int oK = ow.K, omode = ow.mode, oS = mk_uni(od.S), oKR = mk_uni(od.KR);
    const int osubs = q0.subs, oxsrc = mk_uni(od.xsrc);
    const float* oX = mk_uni(od.X);
    const uint16_t* ogamma = mk_uni(od.gamma);
    const int M = a.M;
    const int s = q0.s, g = q0.g, gs = q0.gs;
    const int k0 = q0.k0, KR = oKR, ldk = KR + 8;
    const int nsub = q0.nsub;
    if (nsub == 0) return;
    uint16_t* xh = (uint16_t*)smem;
    uint16_t* xl = xh + (size_t)M * ldk;
    float* red = (float*)(xl + (size_t)M * ldk);  // [2][8][256] wave partial tiles
    float* res = red + 2 * kNW * 256;             // [nsub][256] reduced tiles
    const int n = lane & 15, q = lane >> 4;
    const int wpu = q0.wpu, groups = q0.groups;
    const int kw0 = q0.kw0;
    const int nround = (nsub + groups - 1) / groups;
    // The first kMkPreSteps slices of the first weight unit were requested before this call
    // (during the grid barrier); the rest of it, then the activation rows, follow.
    {
        int st0;
        const uint16_t* p0 = mk_uptr(a, q0, 0, n, q, lane, st0);
        mk_issue<kMkPreSteps, 8>(bf, p0, st0);
    }
    asm volatile("" ::: "memory");
    float* ssq = red + 2048;  // [kMkMaxRows][8] wave partials of the rows' sums of squares
    // Epilogue inputs that come from memory (output row map, residual, RoPE factors) for this
    // workgroup's first kPreTiles tiles, requested together with the activation rows.  Element
    // (m, c) of a tile belongs to thread 16 m + c of the first 256.
    const int em = tid >> 4, ec = tid & 15;
    const int ntile = nsub / osubs;
    const int oldy = mk_uni(od.ldy), ores_embed = mk_uni(od.res_embed);
    const float* oxres = mk_uni(od.xres);
    const int32_t* oout_map = mk_uni(od.out_map);
    constexpr int kPreTiles = 2;
    float pre0[kPreTiles] = {0.f, 0.f}, pre1[kPreTiles] = {0.f, 0.f};
    int orow = em;
    if (em < M) {
        if (omode == kEpiStore) {
            if (oout_map) orow = mk_ldi(oout_map + em);
        } else if (omode == kEpiAdd) {
            if (!ores_embed) {
#pragma unroll
                for (int jt = 0; jt < kPreTiles; ++jt)
                    if (jt < ntile) pre0[jt] = mk_ldg(oxres + (size_t)em * oldy + (g + jt * gs) * 16 + ec);
            }
        } else if (omode == kEpiQkv) {
            const int pos = rp.pos[em], pp = pos < 0 ? 0 : pos, half = a.hd / 2, per_head = a.hd / 16;
#pragma unroll
            for (int jt = 0; jt < kPreTiles; ++jt) {
                int lt = g + jt * gs;
                if (jt < ntile && lt < ow.st0 + ow.st1) {  // Q and K tiles are rotated
                    if (lt >= ow.st0) lt -= ow.st0;
                    const int i = 8 * (lt % per_head) + (ec & 7);
                    pre0[jt] = mk_ldg(a.rcos + (size_t)pp * half + i);
                    pre1[jt] = mk_ldg(a.rsin + (size_t)pp * half + i);
                }
            }
        }
    }
    // Stage rows in passes of eight: x (times the gain) as a bf16 hi/lo pair in LDS.  Each thread
    // reads the gain of its own columns (bf16 ones when the phase has no norm).
    const int n4 = KR / 4;
    uint2 gw[2];
#pragma unroll
    for (int jc = 0; jc < 2; ++jc) {
        const int c = tid + 512 * jc;
        gw[jc] = make_uint2(0x3f803f80u, 0x3f803f80u);
        if (ogamma && c < n4) {
            const mk_u2 w = *(mk_gu2p)(ogamma + k0 + 4 * c);
            gw[jc] = make_uint2(w.x, w.y);
        }
    }
    if (oxsrc == kMkXAttn) {
        // The rows are attention outputs still split into span partials (output, span max, span
        // sum per row, head and span): each thread merges its 4 columns over the spans its row
        // sees, all spans' partials requested at once (up to 16 per round trip), then stages them.
        const int HD = a.hd, ns = mk_uni(od.nsplit);
        for (int m = 0; m < M; ++m) {
            const int pos = rp.pos[m];
            const int nl = pos >= 0 ? min(ns, pos / kMkSpan + 1) : 0;
            float sqm = 0.f;
            for (int c = tid; c < n4 && tid < kNT; c += kNT) {
                const int kk = k0 + 4 * c, h = kk / HD, d = kk % HD;
                float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
                const float* pb = oX + ((size_t)m * a.H + h) * ns * (HD + 4);
                float Mx = -INFINITY, L = 0.f;
                float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int s0 = 0; s0 < nl; s0 += 16) {
                    float4 v[16];
                    float2 ml[16];
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const float* e2 = pb + (size_t)min(s0 + i, nl - 1) * (HD + 4);
                        v[i] = mk_ldg4(e2 + d);
                        ml[i] = mk_ldg2(e2 + HD);
                    }
                    mk_fold16(v, ml, nl - s0, Mx, L, O);
                }
                if (L > 0.f) {
                    const float inv = 1.f / L;
                    x = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
                }
                const mk_f2 a0 = {x.x, x.y}, a1 = {x.z, x.w};
                const mk_bf16x2 h0 = __builtin_convertvector(a0, mk_bf16x2), h1 = __builtin_convertvector(a1, mk_bf16x2);
                const mk_bf16x2 l0 = __builtin_convertvector(a0 - __builtin_convertvector(h0, mk_f2), mk_bf16x2);
                const mk_bf16x2 l1 = __builtin_convertvector(a1 - __builtin_convertvector(h1, mk_f2), mk_bf16x2);
                *(uint2*)(xh + (size_t)m * ldk + 4 * c) = make_uint2(__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1));
                *(uint2*)(xl + (size_t)m * ldk + 4 * c) = make_uint2(__builtin_bit_cast(uint32_t, l0), __builtin_bit_cast(uint32_t, l1));
                sqm += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
            }
            sqm = mk_wsum(sqm);
            if (lane == 0 && wave < kNW) ssq[m * kNW + wave] = sqm;
        }
    } else {
        for (int m0 = 0; m0 < M; m0 += 8) {
            float4 xv[8][2];
            if (oxsrc == kMkXEmbed) {
    #pragma unroll
                for (int mm = 0; mm < 8; ++mm)
    #pragma unroll
                    for (int jc = 0; jc < 2; ++jc) {
                        const int m = m0 + mm, c = tid + 512 * jc;
                        xv[mm][jc] = make_float4(0.f, 0.f, 0.f, 0.f);
                        if (m < M && tid < kNT && c < n4) {
                            const int cc = k0 + 4 * c;
                            xv[mm][jc] = make_float4(mk_embed_at(a, rp, m, cc), mk_embed_at(a, rp, m, cc + 1),
                                                     mk_embed_at(a, rp, m, cc + 2), mk_embed_at(a, rp, m, cc + 3));
                        }
                    }
            } else {
                // every row's loads are issued before any is used: no per-element branches (rows
                // past M and columns past the range re-read the last one; they are not staged)
                const int nr = min(8, M - m0), nj = n4 > 512 ? 2 : 1;
                const int rr = nr <= 1 ? 1 : nr <= 2 ? 2 : nr <= 4 ? 4 : 8;
                if (nj == 1) {
                    if (rr == 1) mk_xload<1, 1>(xv, oX, m0, M, oK, k0, n4, tid);
                    else if (rr == 2) mk_xload<2, 1>(xv, oX, m0, M, oK, k0, n4, tid);
                    else if (rr == 4) mk_xload<4, 1>(xv, oX, m0, M, oK, k0, n4, tid);
                    else mk_xload<8, 1>(xv, oX, m0, M, oK, k0, n4, tid);
                } else {
                    if (rr == 1) mk_xload<1, 2>(xv, oX, m0, M, oK, k0, n4, tid);
                    else if (rr == 2) mk_xload<2, 2>(xv, oX, m0, M, oK, k0, n4, tid);
                    else if (rr == 4) mk_xload<4, 2>(xv, oX, m0, M, oK, k0, n4, tid);
                    else mk_xload<8, 2>(xv, oX, m0, M, oK, k0, n4, tid);
                }
            }
            float sq[8];
    #pragma unroll
            for (int mm = 0; mm < 8; ++mm) {
                const int m = m0 + mm;
                sq[mm] = 0.f;
                if (m >= M) continue;
    #pragma unroll
                for (int jc = 0; jc < 2; ++jc) {
                    const int c = tid + 512 * jc;
                    if (tid < kNT && c < n4) {
                        const float4 v = xv[mm][jc];
                        const uint2 gg = gw[jc];
                        const mk_f2 a0 = {v.x * __uint_as_float(gg.x << 16), v.y * __uint_as_float(gg.x & 0xffff0000u)};
                        const mk_f2 a1 = {v.z * __uint_as_float(gg.y << 16), v.w * __uint_as_float(gg.y & 0xffff0000u)};
                        const mk_bf16x2 h0 = __builtin_convertvector(a0, mk_bf16x2), h1 = __builtin_convertvector(a1, mk_bf16x2);
                        const mk_bf16x2 l0 = __builtin_convertvector(a0 - __builtin_convertvector(h0, mk_f2), mk_bf16x2);
                        const mk_bf16x2 l1 = __builtin_convertvector(a1 - __builtin_convertvector(h1, mk_f2), mk_bf16x2);
                        *(uint2*)(xh + (size_t)m * ldk + 4 * c) =
                            make_uint2(__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1));
                        *(uint2*)(xl + (size_t)m * ldk + 4 * c) =
                            make_uint2(__builtin_bit_cast(uint32_t, l0), __builtin_bit_cast(uint32_t, l1));
                        sq[mm] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
                    }
                }
            }
            // the rows' wave sums are independent DPP chains
    #pragma unroll
            for (int mm = 0; mm < 8; ++mm)
                if (m0 + mm < M) sq[mm] = mk_wsum(sq[mm]);
    #pragma unroll
            for (int mm = 0; mm < 8; ++mm)
                if (m0 + mm < M && lane == 0 && wave < kNW) ssq[(m0 + mm) * kNW + wave] = sq[mm];
        }
    }
    __syncthreads();
    if (tid < M) {
        float tsum = 0.f;
        for (int ww = 0; ww < kNW; ++ww) tsum += ssq[tid * kNW + ww];
        inv_rms[tid] = ogamma ? rsqrtf(tsum / (float)oK + a.eps) : 1.0f;
    }
    __syncthreads();

    // ---- streaming loop: one unit per wave in flight, partial tiles summed every two rounds ----
    const int arow = n < M ? n : M - 1;  // rows >= M repeat row M-1; their outputs are discarded
    const uint16_t* ahp = xh + (size_t)arow * ldk + kw0 + 16 * q;
    const uint16_t* alp = xl + (size_t)arow * ldk + kw0 + 16 * q;
    // Activation fragments are read from LDS two slices at a time, all eight requests ahead of
    // the slices' eight MFMAs (left to itself the scheduler waits on every single read).
    auto mma = [&]() {
        mk_f4 acc = {0.f, 0.f, 0.f, 0.f}, acc2 = acc;
#pragma unroll
        for (int s0 = 0; s0 < 8; s0 += 2) {
            mk_bf16x8 ah[4], al[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int st = s0 + (i >> 1), h = i & 1;
                ah[i] = *(const mk_bf16x8*)(ahp + st * 64 + 8 * h);
                al[i] = *(const mk_bf16x8*)(alp + st * 64 + 8 * h);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int st = s0 + (i >> 1), h = i & 1;
                const mk_bf16x8 b = __builtin_bit_cast(mk_bf16x8, bf.w[st][h]);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[i], b, acc, 0, 0, 0);
                acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], b, acc2, 0, 0, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // the 8 LDS reads
            __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);  // then the 8 MFMAs
        }
        return acc + acc2;
    };
    auto put = [&](const mk_f4& v, int slot) {
#pragma unroll
        for (int r = 0; r < 4; ++r) red[(slot * kNW + wave) * 256 + (4 * q + r) * 16 + n] = v[r];
    };
    auto reduce = [&](int r0, int nr) {
        __syncthreads();
        for (int e = tid; e < nr * groups * 256 && tid < kNT; e += kNT) {
            const int i = e / (groups * 256), gg = (e / 256) % groups, c = e & 255;
            const int u = (r0 + i) * groups + gg;
            if (u < nsub) {
                // all eight wave slots are read at once (slots past the unit's waves are dropped)
                float rv[kNW];
#pragma unroll
                for (int ww = 0; ww < kNW; ++ww) rv[ww] = red[(i * kNW + ((gg * wpu + ww) & (kNW - 1))) * 256 + c];
                float x = 0.f;
#pragma unroll
                for (int ww = 0; ww < kNW; ++ww) x += ww < wpu ? rv[ww] : 0.f;
                res[u * 256 + c] = x * inv_rms[c >> 4];
            }
        }
        __syncthreads();
    };
    int r = 0;
    for (; r + 1 < nround; ++r) {
        mk_f4 acc = {0.f, 0.f, 0.f, 0.f};
        if (wave < kNW) acc = mma();
        if (wave < kNW) {
            int st1;
            const uint16_t* p1 = mk_uptr(a, q0, r + 1, n, q, lane, st1);
            mk_issue(bf, p1, st1);
        }
        if (wave < kNW) put(acc, r & 1);
        if (r & 1) reduce(r - 1, 2);
    }
    {
        mk_f4 acc = {0.f, 0.f, 0.f, 0.f};
        if (wave < kNW) acc = mma();
        if (wave < kNW) put(acc, r & 1);
    }
    if (r & 1) reduce(r - 1, 2);
    else reduce(r, 1);

    // ---- epilogue: element (m, c) of a tile is held by thread 16 m + c of the first 256 ----
    const int olayer = mk_uni(od.layer);
    float* oY = mk_uni(od.Y);
    float* oss_out = mk_uni(od.ss_out);
    float* oqout = mk_uni(od.qout);
    auto epilogue = [&](int jt, float v0, float v1) {
        const int tile = g + jt * gs;
        // every thread of the first 256 calls this (sums of squares need whole 16-lane groups)
        const bool valid = em < M;
        if (omode == kEpiStore) {
            if (valid && orow >= 0) mk_stf(oY + (size_t)orow * oldy + tile * 16 + ec, v0);
        } else if (omode == kEpiAdd) {
            float nv = 0.f;
            if (valid) {
                const int col = tile * 16 + ec;
                const float res0 = ores_embed ? mk_embed_at(a, rp, em, col)
                                   : jt < kPreTiles ? (jt == 0 ? pre0[0] : pre0[1])
                                                    : mk_ldg(oxres + (size_t)em * oldy + col);
                nv = res0 + v0;
                if constexpr (UB) {
                    // steering bias after the MLP (the down projection's phase carries it)
                    const float* oub = mk_uni(od.ubias);
                    if (oub) nv += mk_ldg(oub + (size_t)rp.seq[em] * mk_uni(od.ub_ld) + col);
                }
                mk_stf(oY + (size_t)em * oldy + col, nv);
            }
            if (oss_out) {
                float sq = nv * nv;
#pragma unroll
                for (int off = 8; off > 0; off >>= 1) sq += __shfl_xor(sq, off, 16);
                if (valid && ec == 0) mk_stf(oss_out + (size_t)em * (oldy / 16) + tile, sq);
            }
        } else if (omode == kEpiSwiglu) {
            // MLP steering: the sequence's bias for this layer joins the up projection (eq. (2));
            // compiled only into the instance that runs steered drafter steps
            float ub = 0.f;
            if constexpr (UB) {
                const float* oub = mk_uni(od.ubias);
                if (oub && valid)
                    ub = mk_ldg(oub + (size_t)rp.seq[em] * mk_uni(od.ub_ld) +
                                (osubs == 2 ? tile * 16 + ec : tile * 8 + (ec & 7)));
            }
            if (osubs == 2) {
                const float up = UB ? v1 + ub : v1;
                if (valid) mk_stf(oY + (size_t)em * oldy + tile * 16 + ec, silu(v0) * up);
            } else {
                // column c < 8 holds gate feature 8 tile + c, column c + 8 its up row
                const float upr = __shfl_xor(v0, 8, 16);
                const float up = UB ? upr + ub : upr;
                if (valid && ec < 8) mk_stf(oY + (size_t)em * oldy + tile * 8 + ec, silu(v0) * up);
            }
        } else {  // Q|K|V: rotate-half RoPE on Q and K, cache append of K and V
            const float partner = __shfl_xor(v0, 8, 16);
            if (!valid) return;
            int seg = 0, lt = tile;
            if (lt >= ow.st0) { lt -= ow.st0; seg = 1; }
            if (seg == 1 && lt >= ow.st1) { lt -= ow.st1; seg = 2; }
            const int per_head = a.hd / 16, half = a.hd / 2;
            const int h = lt / per_head, jj = lt % per_head;
            const int i = 8 * jj + (ec & 7);
            const int dim = ec < 8 ? i : half + i;
            const int pos = rp.pos[em];
            float out = v0;
            if (seg < 2) {
                const int pp = pos < 0 ? 0 : pos;
                float c, sn;
                if (jt < kPreTiles) {
                    c = jt == 0 ? pre0[0] : pre0[1];
                    sn = jt == 0 ? pre1[0] : pre1[1];
                } else {
                    c = mk_ldg(a.rcos + (size_t)pp * half + i);
                    sn = mk_ldg(a.rsin + (size_t)pp * half + i);
                }
                out = ec < 8 ? v0 * c - partner * sn : v0 * c + partner * sn;
            }
            if (seg == 0) {
                mk_stf(oqout + (size_t)em * a.H * a.hd + h * a.hd + dim, out);
            } else if (pos >= 0) {
                const size_t idx =
                    ((((size_t)olayer * a.max_batch + rp.seq[em]) * a.Hkv + h) * a.cap + pos) * a.hd + dim;
                // both cache pointers in registers first: selecting between the adjacent
                // arguments directly indexes a stack copy of them
                float* const kcp = mk_uni(a.kc);
                float* const vcp = mk_uni(a.vc);
                mk_stf((seg == 1 ? kcp : vcp) + idx, out);
            }
        }
    };
    if (oS == 1) {
        for (int jt = 0; jt < ntile; ++jt) {
            if (tid < 256) {
                const float v0 = res[(jt * osubs) * 256 + tid];
                const float v1 = osubs == 2 ? res[(jt * 2 + 1) * 256 + tid] : v0;
                epilogue(jt, v0, v1);
            }
        }
        return;
    }
    // K split over S workgroups: partial tiles, one hand-off for all of this workgroup's tiles
    float* opart = mk_uni(od.part);
    int32_t* ocnt = mk_uni(od.cnt);
    for (int jt = 0; jt < ntile; ++jt) {
        const int tile = g + jt * gs;
        float* pt = opart + ((size_t)tile * oS + s) * osubs * 256;
        if (tid < 256)
            for (int sb = 0; sb < osubs; ++sb) mk_stf(pt + sb * 256 + tid, res[(jt * osubs + sb) * 256 + tid]);
    }
    mk_vmwait();
    __syncthreads();
    if (tid < ntile) {
        const int tile = g + tid * gs;
        const int prev = mk_add(ocnt + tile, 1);
        flags[tid] = prev == oS - 1;
        if (prev == oS - 1) mk_sti(ocnt + tile, 0);
    }
    __syncthreads();
    (void)last_flag;
    for (int jt = 0; jt < ntile; ++jt) {
        if (!flags[jt]) continue;
        const int tile = g + jt * gs;
        const float* pt = opart + (size_t)tile * oS * osubs * 256;
        if (tid < 256) {
            // all S partials are requested before any is added (one memory round trip): the loads
            // are unconditional (ranges past S re-read the last; all S are complete here), the
            // sums take the first S in order
            float p0[8], p1[8];
#pragma unroll
            for (int s0 = 0; s0 < 8; ++s0) p0[s0] = mk_ldg(pt + (size_t)min(s0, oS - 1) * osubs * 256 + tid);
            if (osubs == 2) {
#pragma unroll
                for (int s0 = 0; s0 < 8; ++s0) p1[s0] = mk_ldg(pt + (size_t)min(s0, oS - 1) * 2 * 256 + 256 + tid);
            }
            float v0 = 0.f, v1 = 0.f;
#pragma unroll
            for (int s0 = 0; s0 < 8; ++s0) {
                v0 += s0 < oS ? p0[s0] : 0.f;
                if (osubs == 2) v1 += s0 < oS ? p1[s0] : 0.f;
            }
            epilogue(jt, v0, osubs == 2 ? v1 : v0);
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Attention phase: units (sequence, KV head, group of up to kMkQG query vectors, span of kMkSpan
// positions).  The query vectors of a sequence's rows for a KV head's query heads are numbered
// (row, head) row-major and cut into groups of kMkQG, one vector per wave.  A unit scores its
// group against its span (one lane per position), writes an un-normalised partial (output, max,
// sum), and the last span of a (sequence, KV head, group) to arrive merges all live spans in span
// order.  Positions beyond the group's last query position are never loaded.
//
// Cache rows written by earlier launches do not depend on this launch, so a workgroup requests
// those of its first unit while the grid barrier in front of the phase is still open; only the
// rows this launch appends (positions from the sequence's first row on) and the queries are
// read after it.  A cache line holds one row (hd >= 32 floats), so the early reads never bring a
// line that this launch writes into a cache.
// ---------------------------------------------------------------------------------------------
constexpr int kMkQG = kMkWaves;  // query vectors per attention unit

template <int HD>
struct MkKv {
    static constexpr int F4 = kMkSpan * HD / 4 / kMkThreads;  // float4 of K (and of V) per thread
    float4 k[F4], v[F4];
};

struct MkAttnUnit {
    int sp, kvh, sq, qg, q0, nqu, p0, nvalid, nl, newpos;
};

// Spans any row of the launch sees: units are numbered over these only.
__device__ __forceinline__ int mk_attn_spans(const MkArgs& a, const MkRows& rp, int nsplit) {
    int mx = -1;
    for (int r = 0; r < a.M; ++r) mx = max(mx, rp.pos[r]);
    return mx >= 0 ? min(nsplit, mx / kMkSpan + 1) : 1;
}

__device__ __forceinline__ MkAttnUnit mk_attn_unit(const MkArgs& a, const MkRows& rp, int nsplit, int nspan, int u) {
    MkAttnUnit t;
    const int Gq = a.H / a.Hkv, nq = a.rps * Gq, nqg = (nq + kMkQG - 1) / kMkQG;
    t.sp = u % nspan;
    int r = u / nspan;
    t.qg = r % nqg;
    r /= nqg;
    t.kvh = r % a.Hkv;
    t.sq = r / a.Hkv;
    t.q0 = t.qg * kMkQG;
    t.nqu = min(kMkQG, nq - t.q0);
    int maxq = -1, minq = 0x7fffffff;
    for (int i = 0; i < a.rps; ++i) {
        const int ps = rp.pos[t.sq * a.rps + i];
        if (i >= t.q0 / Gq && i <= (t.q0 + t.nqu - 1) / Gq) maxq = max(maxq, ps);
        if (ps >= 0) minq = min(minq, ps);
    }
    t.p0 = t.sp * kMkSpan;
    t.nvalid = maxq >= t.p0 ? min(kMkSpan, maxq - t.p0 + 1) : 0;
    // live spans of the group (those holding a position one of its queries sees)
    t.nl = maxq >= 0 ? min(nsplit, maxq / kMkSpan + 1) : 0;
    t.newpos = minq;  // first position this launch appends for the sequence
    return t;
}

// K and V rows of a unit's span held by this thread: rows older than the launch (fresh = false)
// or the rows it appends (fresh = true).  Rows past the last valid one re-read it.
template <int HD>
__device__ __forceinline__ void mk_attn_kv(const MkArgs& a, const MkRows& rp, int layer, const MkAttnUnit& t, bool fresh,
                                           MkKv<HD>& kv) {
    if (t.nvalid == 0) return;
    const int tid = mk_tid();
    const size_t head_base = (((size_t)layer * a.max_batch + rp.seq[t.sq * a.rps]) * a.Hkv + t.kvh) * a.cap * HD;
    const float* kg = a.kc + head_base + (size_t)t.p0 * HD;
    const float* vg = a.vc + head_base + (size_t)t.p0 * HD;
#pragma unroll
    for (int i = 0; i < MkKv<HD>::F4; ++i) {
        const int e4 = tid + i * kMkThreads;
        const int j = (e4 * 4) / HD, d = (e4 * 4) % HD;
        const int jj = j < t.nvalid ? j : t.nvalid - 1;
        if ((t.p0 + jj >= t.newpos) == fresh) {
            kv.k[i] = mk_ldg4(kg + (size_t)jj * HD + d);
            kv.v[i] = mk_ldg4(vg + (size_t)jj * HD + d);
        }
    }
}

// Wait until KV head kvh's counter reaches `want` (every Q|K|V tile of that head in this layer has
// been written and counted in); bounded like the grid barrier.
__device__ __forceinline__ void mk_kv_wait(const MkArgs& a, int kvh, unsigned want, long& spins) {
    if (threadIdx.x == kCtl && spins >= 0) {
        while ((int)((unsigned)mk_ld(a.qc + kvh * kMkLine) - want) < 0) {
            if (++spins > kMkSpin) {
                mk_sti(a.err, 1);
                spins = -1;  // give up waiting for the rest of the launch (results invalid)
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
}

template <int HD>
__device__ __forceinline__ void mk_attn_t(const MkArgs& a, const MkPhase& od, const MkRows& rp, char* smem, int* last_flag,
                                          MkKv<HD>& kv, unsigned kv_want, long& spins) {
    struct {
        int nsplit, layer, defer;
        const float* qout;
        float *aout, *apart;
        int32_t* cnt;
    } o;
    o.nsplit = mk_uni(od.nsplit);
    o.layer = mk_uni(od.layer);
    o.defer = mk_uni(od.defer);
    o.qout = mk_uni(od.qout);
    o.aout = mk_uni(od.aout);
    o.apart = mk_uni(od.apart);
    o.cnt = mk_uni(od.cnt);
    const int tid = mk_tid(), lane = tid & 63, wave = tid >> 6;
    const int Gq = a.H / a.Hkv;
    const int nq = a.rps * Gq, nqg = (nq + kMkQG - 1) / kMkQG;
    const int nseq = a.M / a.rps;
    const int nspan = mk_attn_spans(a, rp, o.nsplit);
    const int nunit = nseq * a.Hkv * nqg * nspan;
    constexpr int F4 = MkKv<HD>::F4;
    constexpr int D4 = HD / 4;
    float* qs = (float*)smem;                 // [kMkQG][HD]   pre-scaled queries
    float* ks = qs + kMkQG * HD;              // [kMkSpan][HD+4]
    float* vs = ks + kMkSpan * (HD + 4);      // [kMkSpan][HD]
    float* ps = vs + kMkSpan * HD;            // [kMkQG][kMkSpan] probabilities
    float* mq = ps + kMkSpan * kMkQG;         // [kMkQG] span max
    float* lq = mq + kMkQG;                   // [kMkQG] span sum
    for (int u = blockIdx.x; u < nunit; u += a.G) {
        const MkAttnUnit t = mk_attn_unit(a, rp, o.nsplit, nspan, u);
        const int sp = t.sp, kvh = t.kvh, sq = t.sq, nl = t.nl, nvalid = t.nvalid, q0 = t.q0, nqu = t.nqu;
        if (nl == 0 && sp == 0) {
            // no live position (padding): the outputs are zero
            for (int e = tid; e < nqu * HD; e += kMkThreads) {
                const int qv = q0 + e / HD, d = e % HD;
                mk_stf(o.aout + (size_t)(sq * a.rps + qv / Gq) * a.H * HD + (kvh * Gq + qv % Gq) * HD + d, 0.f);
            }
        }
        if (nvalid == 0) continue;  // dead span: no work and no hand-off
        {
            // rows of this launch (and, past the first unit, all rows) and the queries
            if (u != (int)blockIdx.x) {
                if (kv_want) mk_kv_wait(a, kvh, kv_want, spins);
                mk_attn_kv<HD>(a, rp, o.layer, t, false, kv);
            }
            mk_attn_kv<HD>(a, rp, o.layer, t, true, kv);
            constexpr int Q4 = (kMkQG * D4 + kMkThreads - 1) / kMkThreads;  // float4 of queries per thread
            float4 qv4[Q4];
#pragma unroll
            for (int i = 0; i < Q4; ++i) {
                const int e = tid + i * kMkThreads;
                const int qi = e / D4, d = (e % D4) * 4;
                const int qv = q0 + (qi < nqu ? qi : 0);  // vectors past the group repeat its first
                const int row = sq * a.rps + qv / Gq, h = kvh * Gq + qv % Gq;
                qv4[i] = mk_ldg4(o.qout + (size_t)row * a.H * HD + h * HD + d);
            }
#pragma unroll
            for (int i = 0; i < F4; ++i) {
                const int e4 = tid + i * kMkThreads;
                const int j = (e4 * 4) / HD, d = (e4 * 4) % HD;
                *(float4*)(ks + j * (HD + 4) + d) = kv.k[i];
                *(float4*)(vs + j * HD + d) = kv.v[i];
            }
#pragma unroll
            for (int i = 0; i < Q4; ++i) {
                const int e = tid + i * kMkThreads;
                const float4 v = qv4[i];
                if (e < kMkQG * D4) *(float4*)(qs + 4 * e) = make_float4(v.x * a.scale, v.y * a.scale, v.z * a.scale, v.w * a.scale);
            }
            __syncthreads();
            // scores and probabilities: wave w takes query vector w of the group, lane = position
            if (wave < nqu) {
                // blocks of 32 head dims: all of a block's K and query words are requested from LDS
                // before its products (two accumulators)
                float sc0 = 0.f, sc1 = 0.f;
                const float4* kr = (const float4*)(ks + lane * (HD + 4));
                const float4* qr = (const float4*)(qs + wave * HD);
#pragma unroll 1
                for (int d0 = 0; d0 < D4; d0 += 8) {
                    float4 kx[8], qx[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        kx[i] = kr[d0 + i];
                        qx[i] = qr[d0 + i];
                    }
#pragma unroll
                    for (int i = 0; i < 8; i += 2) {
                        sc0 += qx[i].x * kx[i].x + qx[i].y * kx[i].y + qx[i].z * kx[i].z + qx[i].w * kx[i].w;
                        sc1 += qx[i + 1].x * kx[i + 1].x + qx[i + 1].y * kx[i + 1].y + qx[i + 1].z * kx[i + 1].z +
                               qx[i + 1].w * kx[i + 1].w;
                    }
                }
                const float sc = sc0 + sc1;
                const int qv = q0 + wave;
                const int qp = rp.pos[sq * a.rps + qv / Gq];
                const float v = (lane < nvalid && t.p0 + lane <= qp) ? sc : -INFINITY;
                const float mx = mk_wmax(v);
                const float pr = v == -INFINITY ? 0.f : expf(v - mx);
                const float sm = mk_wsum(pr);
                ps[wave * kMkSpan + lane] = pr;  // [query][position]
                if (lane == 0) {
                    mq[wave] = mx;
                    lq[wave] = sm;
                }
            }
            __syncthreads();
            // un-normalised outputs: a thread per (query vector, head dim), NI vectors kMkThreads / HD
            // apart; a position's probability is a broadcast read, its V element is read once
            constexpr int STEP = kMkThreads / HD;  // vectors between a thread's items
            constexpr int NI = (kMkQG + STEP - 1) / STEP;
            static_assert(NI == 1 || NI * STEP == kMkQG, "a thread's items stay inside the group");
            const int d = tid % HD, qi0 = tid / HD;  // qi0 < STEP
            if (qi0 < nqu) {
                float acc[NI];
#pragma unroll
                for (int i = 0; i < NI; ++i) acc[i] = 0.f;
                // blocks of 16 positions: V elements and probabilities are all requested from LDS
                // before the block's products
#pragma unroll 1
                for (int j0 = 0; j0 < kMkSpan; j0 += 16) {
                    float vv[16];
                    float4 pp[NI][4];
#pragma unroll
                    for (int jj = 0; jj < 16; ++jj) vv[jj] = vs[(j0 + jj) * HD + d];
#pragma unroll
                    for (int i = 0; i < NI; ++i)
#pragma unroll
                        for (int k = 0; k < 4; ++k) pp[i][k] = *(const float4*)(ps + (qi0 + i * STEP) * kMkSpan + j0 + 4 * k);
#pragma unroll
                    for (int i = 0; i < NI; ++i)
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            acc[i] += pp[i][k].x * vv[4 * k];
                            acc[i] += pp[i][k].y * vv[4 * k + 1];
                            acc[i] += pp[i][k].z * vv[4 * k + 2];
                            acc[i] += pp[i][k].w * vv[4 * k + 3];
                        }
                }
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    const int qi = qi0 + i * STEP;
                    if (qi >= nqu) break;
                    const int qv = q0 + qi;
                    const int row = sq * a.rps + qv / Gq, h = kvh * Gq + qv % Gq;
                    if (nl == 1 && !o.defer) {
                        // the only live span: normalise and write the output itself
                        const float l = lq[qi];
                        mk_stf(o.aout + (size_t)row * a.H * HD + h * HD + d, l > 0.f ? acc[i] / l : 0.f);
                    } else {
                        float* pp = o.apart + (((size_t)row * a.H + h) * o.nsplit + sp) * (HD + 4);
                        mk_stf(pp + d, acc[i]);
                        if (d == 0) {
                            mk_stf(pp + HD, mq[qi]);
                            mk_stf(pp + HD + 1, lq[qi]);
                        }
                    }
                }
            }
        }
        if (nl == 1 || o.defer) {
            __syncthreads();  // LDS of this unit is reused by the next
            continue;
        }
        // count in; the last live span of this (sequence, KV head, group) merges the live spans
        mk_vmwait();
        __syncthreads();
        if (tid == 0) {
            int32_t* c = o.cnt + ((size_t)sq * a.Hkv + kvh) * nqg + t.qg;
            const int prev = mk_add(c, 1);
            *last_flag = prev == nl - 1;
            if (prev == nl - 1) mk_sti(c, 0);
        }
        __syncthreads();
        if (*last_flag && tid < nqu * D4) {
            // a thread per (query vector, 4 head dims) requests the partial outputs and the
            // (max, sum) of sixteen spans at once and folds them into a running (max, sum, output)
            const int qv = q0 + tid / D4, d = (tid % D4) * 4;
            const int row = sq * a.rps + qv / Gq, h = kvh * Gq + qv % Gq;
            float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
            if (rp.pos[row] >= 0) {
                const float* pb = o.apart + ((size_t)row * a.H + h) * o.nsplit * (HD + 4);
                float Mx = -INFINITY, L = 0.f;
                float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int s0 = 0; s0 < nl; s0 += 16) {
                    float4 v[16];
                    float2 ml[16];
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const float* e2 = pb + (size_t)min(s0 + i, nl - 1) * (HD + 4);
                        v[i] = mk_ldg4(e2 + d);
                        ml[i] = mk_ldg2(e2 + HD);
                    }
                    mk_fold16(v, ml, nl - s0, Mx, L, O);
                }
                if (L > 0.f) {
                    const float inv = 1.f / L;
                    r = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
                }
            }
            float* op = o.aout + (size_t)row * a.H * HD + h * HD + d;
            mk_stf(op, r.x);
            mk_stf(op + 1, r.y);
            mk_stf(op + 2, r.z);
            mk_stf(op + 3, r.w);
        }
        __syncthreads();
    }
}

// Grid barrier at the start of a phase.  One arrival counter per XCD group (workgroup id mod 8)
// and one release line per group; both only grow (after barrier g of this state, group x's counter
// holds g * (workgroups in group x) and its release line g), and the host passes the number of
// barriers before the launch, so no workgroup reads a starting value that a faster one may already
// have advanced.  A workgroup's control thread adds 1 to its group's counter; the group's last
// arriver writes g to the group's release line; lanes 0..7 of wave 0 poll the eight release lines
// until all hold g.  The polled lines never take atomics (polling the counters themselves, or one
// word per workgroup, measured slower: the polls then contend with the arrivals).
//
// With a weight buffer (projection phases) the phase's first weight unit is requested right after
// the arrival, so that it streams during the barrier.
__device__ __forceinline__ void mk_barrier(const MkArgs& a, int& gen, long& spins, const MkPhase* ph, MkBuf* bf) {
    int32_t* cnt = a.bar;
    int32_t* rel = a.bar + 8 * kMkLine;
    const unsigned g1 = (unsigned)gen + 1u;
    gen = (int)g1;
    if (threadIdx.x == kCtl) {
        const int x = blockIdx.x & 7;
        const unsigned per = (unsigned)(a.G / 8 + (x < a.G % 8 ? 1 : 0));
        const unsigned prev = (unsigned)mk_add(cnt + x * kMkLine, 1);
        if (prev + 1u == g1 * per) mk_sti(rel + x * kMkLine, (int)g1);
    }
    if (bf) {
        const int tid = mk_tid(), lane = tid & 63, wave = tid >> 6;
        const MkGeo q = mk_geo(a, *ph, wave);
        int st;
        const uint16_t* wp = mk_uptr(a, q, 0, lane & 15, lane >> 4, lane, st);
        mk_issue<0, kMkPreSteps>(*bf, wp, st);
    }
    if (threadIdx.x < 64 && spins >= 0) {
        const int l = threadIdx.x;
        for (;;) {
            const bool ok = l >= 8 || (int)((unsigned)mk_ld(rel + l * kMkLine) - g1) >= 0;
            if (__builtin_amdgcn_read_exec() == __ballot(ok)) break;
            if (++spins > kMkSpin) {
                if (l == 0) mk_sti(a.err, 1);
                spins = -1;  // give up waiting for the rest of the launch (results invalid)
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __builtin_amdgcn_s_barrier();
}

// Attention phase with the barrier in front of it: the older cache rows of this workgroup's first
// unit are requested before the release (by waves 1..7 before, by wave 0, which runs the barrier,
// after it, so that its polls do not return behind them).
template <int HD>
__device__ __forceinline__ void mk_attn_phase(const MkArgs& a, const MkPhase& od, const MkRows& rp, char* smem,
                                              int* last_flag, int& gen, long& spins, int p) {
    MkKv<HD> kv;
    const int nsplit = mk_uni(od.nsplit), layer = mk_uni(od.layer);
    const int nq = a.rps * (a.H / a.Hkv);
    const int nspan = mk_attn_spans(a, rp, nsplit);
    const int nunit = (a.M / a.rps) * a.Hkv * ((nq + kMkQG - 1) / kMkQG) * nspan;
    const bool first = (int)blockIdx.x < nunit;
    MkAttnUnit t{};
    if (first) t = mk_attn_unit(a, rp, nsplit, nspan, blockIdx.x);
    const int kvwait = mk_uni(od.kvwait);
    const unsigned want = a.qc_base + (unsigned)(layer + 1) * (unsigned)a.qc_tpk;
    if (first && threadIdx.x >= 64) mk_attn_kv<HD>(a, rp, layer, t, false, kv);
    if (!kvwait) {
        if (p > 0) mk_barrier(a, gen, spins, nullptr, nullptr);
    } else if (first && t.nvalid > 0) {
        mk_kv_wait(a, t.kvh, want, spins);  // only this unit's KV head: no grid barrier
    }
    if (first && threadIdx.x < 64) mk_attn_kv<HD>(a, rp, layer, t, false, kv);
    mk_attn_t<HD>(a, od, rp, smem, last_flag, kv, kvwait ? want : 0u, spins);
}

// One kernel per head dim (64: drafter, 128: verifier), so that each holds one attention
// instantiation: the code of a launch then stays closer to the instruction cache's size.  UB:
// the epilogues add the MLP-steering biases (to up in SwiGLU phases, or after the MLP in the down
// projection's phase; drafter steps with that steering only: the other instances carry no code
// for it).
template <int HD, bool UB>
__global__ __launch_bounds__(kMkThreads) void k_mk(MkArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ MkPhase op_lds[2];
    __shared__ MkRows rp;
    __shared__ float inv_rms[kMkMaxRows];
    __shared__ int flags[64];
    __shared__ int last_flag;
    constexpr int kWords = (int)(sizeof(MkPhase) / 4);
    static_assert(sizeof(MkPhase) % 4 == 0 && kWords <= 64, "phase descriptor larger than one wave");
    mk_plan(a, rp);
    if (threadIdx.x < kWords) ((uint32_t*)&op_lds[0])[threadIdx.x] = mk_ldu((const uint32_t*)&a.prog[0] + threadIdx.x);
    __syncthreads();
    int gen = (int)a.bar_gen;
    long spins = 0;
    if (a.trace && blockIdx.x == 0 && threadIdx.x == kCtl) a.trace[0] = wall_clock64();
    for (int p = 0; p < a.nphase; ++p) {
        // this phase's descriptor stays in LDS; the phase reads the fields it needs
        const MkPhase& o = op_lds[p & 1];
        const int op = mk_uni(o.op);
        // the next descriptor is requested now and reaches LDS after the phase
        uint32_t nw = 0;
        if (threadIdx.x < kWords && p + 1 < a.nphase) nw = mk_ldu((const uint32_t*)&a.prog[p + 1] + threadIdx.x);
        if (op == kMkGemv) {
            MkBuf bf;  // weight unit in flight, per wave
            if (p > 0) {
                mk_barrier(a, gen, spins, &o, &bf);
            } else {
                const int tid = mk_tid(), lane = tid & 63;
                const MkGeo q = mk_geo(a, o, tid >> 6);
                int st;
                const uint16_t* wp = mk_uptr(a, q, 0, lane & 15, lane >> 4, lane, st);
                mk_issue<0, kMkPreSteps>(bf, wp, st);
            }
            mk_gemv<UB>(a, o, rp, smem, inv_rms, flags, &last_flag, bf);
        } else if (op == kMkAttn) {
            mk_attn_phase<HD>(a, o, rp, smem, &last_flag, gen, spins, p);
        }
        mk_vmwait();  // this phase's stores are complete before the workgroup counts in
        if (threadIdx.x < kWords && p + 1 < a.nphase) ((uint32_t*)&op_lds[(p + 1) & 1])[threadIdx.x] = nw;
        __syncthreads();  // next descriptor in LDS; this phase's LDS use is over
        if (threadIdx.x == kCtl && op == kMkGemv && o.kvsig) {
            // Q|K|V tiles of this workgroup are written and complete: count each in on its KV head
            const int st0 = o.seg_tiles[0], st1 = o.seg_tiles[1], ph = a.hd / 16, Gq = a.H / a.Hkv;
            for (int t = blockIdx.x; t < o.tiles; t += a.G) {
                const int kvh = t < st0 ? t / ph / Gq : (t < st0 + st1 ? (t - st0) / ph : (t - st0 - st1) / ph);
                mk_add(a.qc + kvh * kMkLine, 1);
            }
        }
        if (a.trace && blockIdx.x == 0 && threadIdx.x == kCtl && p + 1 < kMkTracePhases) a.trace[p + 1] = wall_clock64();
    }
}

// =============================================================================================
// Host side: phase lists.
// =============================================================================================
namespace {

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

struct MkPlanG {
    int S, KR, wpu;
    size_t lds;
};

// Split of K for a projection of M rows: smallest S with K-range KR a multiple of 512 up to
// kMkMaxKR (8 waves x 512 columns), the staged rows in LDS, and no split for normed inputs
// (their row statistics come from the whole staged row).
MkPlanG mk_plan_gemv(int M, int N, int K, bool norm, int subs) {
    MkPlanG p{0, 0, 0, 0};
    for (int S = 1; S <= 8; S *= 2) {
        if (norm && S > 1) break;
        if (K % S) continue;
        const int KR = K / S;
        if (KR % 512 || KR > kMkMaxKR) continue;
        const int tiles = N / 16;
        const size_t units = (size_t)((tiles * S + kMkMinWG - 1) / kMkMinWG) * subs;  // per workgroup
        const size_t lds = (size_t)M * (KR + 8) * 4 + 2 * kNW * 256 * 4 + units * 1024;
        if (lds > (size_t)kMkLdsBudget) continue;
        p.S = S;
        p.KR = KR;
        p.wpu = KR / 512;
        p.lds = lds;
        return p;
    }
    return p;
}

size_t mk_attn_lds(int hd) {
    return sizeof(float) * ((size_t)kMkQG * hd + (size_t)kMkSpan * (hd + 4) + (size_t)kMkSpan * hd +
                            (size_t)kMkQG * kMkSpan + 2 * kMkQG);
}

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

int mk_nsplit(int cap) { return (cap + kMkSpan - 1) / kMkSpan; }

// Phases of one launch of model m with M rows (rps per sequence); appends to `out` when given.
// Returns false when a shape is not supported.  `lds` receives the largest dynamic LDS.
bool mk_record(const sd2_config& c, const ModelDev& m, bool verifier, int M, int rps, int j, int G, Arena& ar,
               const Workspace* ws, std::vector<MkPhase>* out, size_t* lds, int32_t* cnt, float** final_x,
               float** final_ss, double* bytes_out = nullptr, const float** tap_x = nullptr) {
    double bytes = 0.0;
    const sd2_dims& d = m.dm;
    const int hd = d.d_model / d.n_heads;
    const int L = d.n_layers, H = d.n_heads, Hkv = d.n_kv_heads, F = d.d_ff, dm = d.d_model;
    if (M > kMkMaxRows || M < 1 || Hkv > kMkQcLines) return false;
    if (rps * (H / Hkv) > kMkMaxNq) return false;
    // head dims 64 and 128 only: each instantiation adds ~15 KB to a kernel that already exceeds
    // the instruction cache (other head dims take the per-operation path)
    if (hd != 64 && hd != 128) return false;
    const int nsplit = mk_nsplit(c.max_seq_len);
    size_t mx = mk_attn_lds(hd);
    auto gemv = [&](int mode, int N, int K, const void* gamma, bool norm, int subs, MkPhase& ph) -> bool {
        MkPlanG pl = mk_plan_gemv(M, N, K, norm, subs);
        if (!pl.S || (G > 0 && G % pl.S)) return false;
        ph.op = kMkGemv;
        ph.mode = mode;
        ph.K = K;
        ph.tiles = N / 16;
        ph.S = pl.S;
        ph.KR = pl.KR;
        ph.wpu = pl.wpu;
        ph.subs = subs;
        ph.gamma = (const uint16_t*)gamma;
        ph.cnt = cnt;
        if (pl.S > 1) ph.part = ar.take<float>((size_t)ph.tiles * pl.S * subs * 256);
        mx = std::max(mx, pl.lds);
        bytes += (double)ph.tiles * 16 * K * 2.0 * subs;
        return N % 16 == 0;
    };
    const void* const* W = m.layer;
    float* x_prev = nullptr;  // null: the embedding rows (+ steering)
    for (int l = 0; l < L; ++l) {
        const void* const* Wl = W + (size_t)l * 9;
        float* q = ar.take<float>((size_t)M * H * hd);
        float* att = ar.take<float>((size_t)M * H * hd);
        float* xa = ar.take<float>((size_t)M * dm);
        float* hbuf = ar.take<float>((size_t)M * F);
        float* xf = ar.take<float>((size_t)M * dm);
        float* apart = ar.take<float>((size_t)M * H * nsplit * (hd + 4));
        float* ss = (l == L - 1) ? ar.take<float>((size_t)M * (dm / 16)) : nullptr;
        MkPhase qkv{};
        if (!gemv(kEpiQkv, (H + 2 * Hkv) * hd, dm, Wl[kAttnNorm], true, 1, qkv)) return false;
        qkv.nseg = 3;
        qkv.W[0] = (const uint16_t*)Wl[kWq];
        qkv.W[1] = (const uint16_t*)Wl[kWk];
        qkv.W[2] = (const uint16_t*)Wl[kWv];
        qkv.seg_tiles[0] = H * hd / 16;
        qkv.seg_tiles[1] = Hkv * hd / 16;
        qkv.seg_tiles[2] = Hkv * hd / 16;
        qkv.xsrc = x_prev ? kMkXBuf : kMkXEmbed;
        qkv.kvsig = 1;
        qkv.X = x_prev;
        qkv.qout = q;
        qkv.layer = l;
        MkPhase at{};
        at.op = kMkAttn;
        at.layer = l;
        at.nsplit = nsplit;
        at.qout = q;
        at.aout = att;
        at.apart = apart;
        at.cnt = cnt;
        at.kvwait = 1;  // waits for its KV head's Q|K|V tiles only (the Q|K|V phase counts them in)
        // Few rows (drafter steps): the O projection merges the span partials while it stages its
        // input, so no attention workgroup waits to merge; each O workgroup then reads all rows'
        // partials (at most 256 KB, mostly from L2).
        at.defer = (size_t)M * H * nsplit * (hd + 4) * sizeof(float) <= 256 * 1024 ? 1 : 0;
        MkPhase o{};
        if (!gemv(kEpiAdd, dm, H * hd, nullptr, false, 1, o)) return false;
        if (at.defer && o.S != 1) at.defer = 0;
        o.nseg = 1;
        o.W[0] = (const uint16_t*)Wl[kWo];
        o.X = at.defer ? apart : att;
        o.xsrc = at.defer ? kMkXAttn : kMkXBuf;
        o.nsplit = nsplit;
        o.xres = x_prev;
        o.res_embed = x_prev ? 0 : 1;
        o.Y = xa;
        o.ldy = dm;
        MkPhase gu{};
        // Tiles of 16 features with a gate and an up sub-tile when F / 16 tiles spread evenly over
        // the workgroups; else tiles of 8 gate + 8 up rows (2F / 16 of them: twice as many, so the
        // last round is not left to half of the workgroups)
        const bool pair_tiles = G > 0 && (F / 16) % G == 0;
        if (pair_tiles) {
            if (!gemv(kEpiSwiglu, F, dm, Wl[kFfnNorm], true, 2, gu)) return false;
        } else if (F % 8 || !gemv(kEpiSwiglu, 2 * F, dm, Wl[kFfnNorm], true, 1, gu)) {
            return false;
        }
        gu.nseg = pair_tiles ? 2 : 1;
        gu.W[0] = (const uint16_t*)Wl[kWg];
        gu.W[1] = (const uint16_t*)Wl[kWu];
        gu.X = xa;
        gu.Y = hbuf;
        gu.ldy = F;
        if (!verifier && ws && c.steering == SD2_STEER_MLP) {
            gu.ubias = ws->ubias + (size_t)l * F;
            gu.ub_ld = L * F;
        }
        MkPhase dn{};
        if (!gemv(kEpiAdd, dm, F, nullptr, false, 1, dn)) return false;
        dn.nseg = 1;
        dn.W[0] = (const uint16_t*)Wl[kWd];
        dn.X = hbuf;
        dn.xres = xa;
        dn.Y = xf;
        dn.ldy = dm;
        dn.ss_out = ss;
        if (!verifier && ws && c.steering == SD2_STEER_MLP_OUT) {
            dn.ubias = ws->ubias;
            dn.ub_ld = dm;
        }
        if (out) {
            out->push_back(qkv);
            out->push_back(at);
            out->push_back(o);
            out->push_back(gu);
            out->push_back(dn);
        }
        x_prev = xf;
        // MLP steering taps: residual after blocks L-2, floor(L/2), 3 (from 1); each layer's
        // residual has its own buffer, so the rows stay readable after the launch
        if (tap_x) {
            const int tl[3] = {L - 3, L / 2 - 1, 2};
            for (int sl = 0; sl < 3; ++sl)
                if (tl[sl] == l) tap_x[sl] = xf;
        }
        if (l == L - 1) {
            if (final_x) *final_x = xf;
            if (final_ss) *final_ss = ss;
        }
    }
    MkPhase lm{};
    if (!gemv(kEpiStore, d.vocab, dm, m.final_norm, true, 1, lm)) return false;
    lm.nseg = 1;
    lm.W[0] = (const uint16_t*)m.lm_head;
    lm.gamma = (const uint16_t*)m.final_norm;
    lm.X = x_prev;
    lm.ldy = d.vocab;
    if (ws) {
        lm.Y = verifier ? ws->logits_v : ws->logits_d;
        lm.out_map = verifier ? nullptr : ws->lm_map_d + (size_t)(j - 1) * 2 * c.max_batch;
    }
    if (out) out->push_back(lm);
    if (lds) *lds = std::max(*lds, mx);
    if (bytes_out) *bytes_out = bytes;
    return true;
}

}  // namespace

// Largest batch for which both launch kinds are supported (0: none).
int mk_max_batch(const sd2_config& c) {
    // the conditional bias runs one kernel per operation
    if (c.dtype != SD2_BF16 || c.steering == SD2_STEER_MLP_COND) return 0;
    ModelDev mv{}, md{};
    mv.dm = c.verifier;
    md.dm = c.drafter;
    for (int b = std::min(c.max_batch, kMkMaxRows); b >= 1; --b) {
        Arena ar{nullptr, 0};
        if (mk_record(c, md, false, 2 * b, 2, 1, 0, ar, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) &&
            mk_record(c, md, false, b, 1, 2, 0, ar, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) &&
            mk_record(c, mv, true, b * (c.k + 1), c.k + 1, 0, 0, ar, nullptr, nullptr, nullptr, nullptr, nullptr,
                      nullptr))
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
        mk_record(c, md, false, 2 * batch, 2, 1, 0, ar, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
        mx = std::max(mx, ar.off);
    }
    {
        Arena ar{nullptr, 0};
        mk_record(c, mv, true, batch * (c.k + 1), c.k + 1, 0, 0, ar, nullptr, nullptr, nullptr, nullptr, nullptr,
                  nullptr);
        mx = std::max(mx, ar.off);
    }
    return mx;
}

int mk_phase_count(const sd2_config& c) {
    return c.k * (5 * c.drafter.n_layers + 1) + 5 * c.verifier.n_layers + 1;
}

size_t mk_counter_ints(const sd2_config& c) {
    const int v = c.verifier.vocab / 16 + 1;
    const int f = std::max(c.verifier.d_ff, c.drafter.d_ff) / 16 + 1;
    // attention: one counter per (sequence, KV head, group of query vectors)
    const int kv = kMkMaxRows * std::max(c.verifier.n_kv_heads, c.drafter.n_kv_heads) * (kMkMaxNq / kMkQG);
    return (size_t)std::max(std::max(v, f), kv);
}

__global__ void k_mk_init(uint16_t* ones, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) ones[i] = 0x3f80;  // bf16 1.0
}

void mk_init_buffers(Engine& e) {
    e.mk.bar_gen = 0;  // the barrier and KV-head counters are zero in a fresh workspace
    e.mk.qc_total[0] = e.mk.qc_total[1] = 0;
    if (!e.mk.ones) return;
    k_mk_init<<<(kMkMaxKR + 255) / 256, 256, 0, e.stream>>>(e.mk.ones, kMkMaxKR);
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
    if (cus < kMkMinWG || cus % 8) return false;  // LDS plans assume >= kMkMinWG workgroups
    s.G = cus;
    std::vector<MkPhase> prog;
    size_t lds = 0;
    const sd2_config& c = e.cfg;
    for (int j = 1; j <= c.k; ++j) {
        Arena ar{s.arena, 0};
        s.off[j] = (int)prog.size();
        if (!mk_record(c, e.md, false, j == 1 ? 2 * batch : batch, j == 1 ? 2 : 1, j, s.G, ar, &e.ws, &prog, &lds,
                       s.cnt, nullptr, nullptr, &s.bytes[j]) ||
            ar.off > s.arena_bytes)
            return false;
        s.n[j] = (int)prog.size() - s.off[j];
    }
    {
        Arena ar{s.arena, 0};
        s.off[0] = (int)prog.size();
        if (!mk_record(c, e.mv, true, batch * (c.k + 1), c.k + 1, 0, s.G, ar, &e.ws, &prog, &lds, s.cnt, &s.final_x,
                       &s.final_ss, &s.bytes[0], s.tap_x) ||
            ar.off > s.arena_bytes)
            return false;
        s.n[0] = (int)prog.size() - s.off[0];
    }
    if ((int)prog.size() > s.prog_cap) return false;
    s.lds = lds;
    for (const void* fn : {(const void*)k_mk<64, false>, (const void*)k_mk<128, false>, (const void*)k_mk<64, true>,
                           (const void*)k_mk<128, true>})
        if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) return false;
    int occ = 0;
    for (const void* fn : {(const void*)k_mk<64, false>, (const void*)k_mk<128, false>, (const void*)k_mk<64, true>,
                           (const void*)k_mk<128, true>})
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, kMkThreads, lds) != hipSuccess || occ < 1) return false;
    if (hipMemcpyAsync(s.prog, prog.data(), sizeof(MkPhase) * prog.size(), hipMemcpyHostToDevice, e.stream) !=
        hipSuccess)
        return false;
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
    // MLP steering biases the up projections instead; an unsteered drafter adds nothing
    a.add_steer = ver || e.mlp || !e.w_steer ? 0 : 1;
    a.kc = m.kc;
    a.vc = m.vc;
    a.rcos = m.rope_cos;
    a.rsin = m.rope_sin;
    a.dummy = s.dummy;
    a.ones = s.ones;
    a.bar = s.bar;
    a.bar_gen = s.bar_gen;
    a.qc = s.qc + (size_t)(ver ? 0 : 1) * kMkQcLines * kMkLine;
    a.qc_base = s.qc_total[ver ? 0 : 1];
    a.qc_tpk = (m.dm.n_heads / m.dm.n_kv_heads + 2) * (m.hd / 16);
    a.err = s.err;
    a.trace = (e.prof_on && s.trace) ? s.trace + (size_t)j * kMkTracePhases : nullptr;
    a.G = s.G;
    void* args[] = {&a};
    ProfEntry* pe = prof_slot(&e, kProfProgram, s.bytes[j]);
    if (pe) (void)hipEventRecord(pe->a, e.stream);
    const bool ub = !ver && e.mlp;
    const void* fn = m.hd == 64 ? (ub ? (const void*)k_mk<64, true> : (const void*)k_mk<64, false>)
                                : (ub ? (const void*)k_mk<128, true> : (const void*)k_mk<128, false>);
    hipError_t err = hipLaunchCooperativeKernel(fn, dim3(s.G), dim3(kMkThreads), args, s.lds, e.stream);
    if (pe) {
        (void)hipEventRecord(pe->b, e.stream);
        prof_commit(&e);
    }
    if (err == hipSuccess) {
        // one grid barrier per phase after the first, except the attention phases (one per layer)
        s.bar_gen += (uint32_t)(s.n[j] - 1 - m.dm.n_layers);
        s.qc_total[ver ? 0 : 1] += (uint32_t)(m.dm.n_layers * a.qc_tpk);
    }
    return err;
}

}  // namespace sd2
