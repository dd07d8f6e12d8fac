// Grouped-query causal attention over the fp32 KV cache for a block of query rows.
//
// Split over cache positions (flash-decoding): one workgroup owns up to 32 query vectors of one
// sequence -- either one query head for a tile of rows (small batches: more workgroups, the KV
// head shared through L2) or all query heads of one KV head (large batches: each cached K/V
// row read once) -- and one span of kSplit cache positions.  It walks its span in chunks of 64
// positions with an online softmax (running max, running sum, rescaled output), keeping the
// next chunk's K/V in flight in registers while the current chunk is scored from LDS, and
// writes an un-normalised partial (output, max, sum); the last span to finish for a set of
// query vectors merges all spans in span order (see arrive_last).  The causal mask is key position <= query position; rows
// with position -1 are inactive and produce zeros.  Workgroups of one KV head are placed on
// the same XCD (workgroup ids are dealt round-robin over the 8 XCDs), so a KV head is fetched
// into one L2 only.
#include <math.h>

#include <algorithm>

#include <hip/hip_ext.h>

#include "device_common.h"
#include "engine.h"

namespace sd2 {

constexpr int kAttnCL = 64;   // cache positions per chunk
constexpr int kSplit = 128;   // cache positions per workgroup
constexpr int kAttnQT = 32;   // query vectors per workgroup
constexpr int kAttnT = 256;
constexpr int kXcds = 8;

typedef float f4_t __attribute__((ext_vector_type(4)));

struct AttnArgs {
    const float* q;
    int q_stride;
    const float *kc, *vc;
    float* out;
    const int32_t* row_pos;
    int rps, H, Hkv, hd, cap, max_batch, layer;
    int hp;     // query heads per workgroup: 1 or H/Hkv
    int nrt;    // row tiles per (sequence, head group)
    int ngrp;   // number of (sequence, KV head, row tile) groups
    int nsplit; // position spans per group
    float scale;
    float* part;     // [row][head][nsplit][HD + 2]
    int32_t* cnt;    // one arrival counter per workgroup of the split-free grid
};

// Wave-wide max and sum with DPP steps (quad permutes, row mirrors, row broadcasts), every lane
// active; the result is read from lane 63 and is uniform.  xor shuffles through LDS took six
// dependent LDS round trips per reduction.
template <int CTRL, int ROWS>
__device__ __forceinline__ float at_dpp(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v),
                                                                 CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float at_wmax(float v) {
    v = fmaxf(v, at_dpp<0xB1, 0xf>(v, v));   // quad_perm [1,0,3,2]
    v = fmaxf(v, at_dpp<0x4E, 0xf>(v, v));   // quad_perm [2,3,0,1]
    v = fmaxf(v, at_dpp<0x141, 0xf>(v, v));  // row_half_mirror
    v = fmaxf(v, at_dpp<0x140, 0xf>(v, v));  // row_mirror
    v = fmaxf(v, at_dpp<0x142, 0xa>(v, v));  // row_bcast:15 into rows 1 and 3
    v = fmaxf(v, at_dpp<0x143, 0xc>(v, v));  // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float at_wsum(float v) {
    v += at_dpp<0xB1, 0xf>(0.f, v);
    v += at_dpp<0x4E, 0xf>(0.f, v);
    v += at_dpp<0x141, 0xf>(0.f, v);
    v += at_dpp<0x140, 0xf>(0.f, v);
    v += at_dpp<0x142, 0xa>(0.f, v);
    v += at_dpp<0x143, 0xc>(0.f, v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Request chunk c of K and V (positions past maxpos re-read the last valid row; they are masked).
template <int HD, int F4>
__device__ __forceinline__ void fetch_chunk(f4_t (&pk)[F4], f4_t (&pv)[F4], const float* kg, const float* vg,
                                            int c, int maxpos, int tid) {
#pragma unroll
    for (int i = 0; i < F4; ++i) {
        int e4 = tid + i * kAttnT;  // float4 index within the chunk
        int pos = c * kAttnCL + (e4 * 4) / HD;
        int pp = pos <= maxpos ? pos : maxpos;
        pk[i] = *(const f4_t*)(kg + (size_t)pp * HD + (e4 * 4) % HD);
        pv[i] = *(const f4_t*)(vg + (size_t)pp * HD + (e4 * 4) % HD);
    }
}

template <int HD, int QT>
__global__ __launch_bounds__(kAttnT) void k_attn(AttnArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    __shared__ int qpos[QT];
    __shared__ int qrow[QT];
    __shared__ int qhead[QT];
    __shared__ float mrun[QT], lrun[QT], rescale[QT];
    __shared__ int maxpos_s;
    __shared__ int last_flag;
    const int tid = threadIdx.x;
    const int G = a.H / a.Hkv;
    const int members = G / a.hp;  // workgroups per group
    // XCD-aware decode: the `members` workgroups of a group share wg % 8
    const int wg = blockIdx.x / a.nsplit;
    const int sp = blockIdx.x % a.nsplit;
    const int gi = (wg / (kXcds * members)) * kXcds + wg % kXcds;
    const int mi = (wg / kXcds) % members;
    if (gi >= a.ngrp) return;
    const int rt = gi % a.nrt;
    const int kvh = (gi / a.nrt) % a.Hkv;
    const int b = gi / (a.nrt * a.Hkv);
    const int hbase = kvh * G + mi * a.hp;
    const int rows_per_tile = QT / a.hp;
    const int r0 = rt * rows_per_tile;
    const int nrows = min(rows_per_tile, a.rps - r0);
    const int nq = nrows * a.hp;

    float* qs = sm;                          // [QT][HD]   (pre-scaled queries)
    float* ks = qs + QT * HD;           // [CL][HD+1]
    float* vs = ks + kAttnCL * (HD + 1);     // [CL][HD]
    float* ps = vs + kAttnCL * HD;           // [QT][CL]

    if (tid == 0) maxpos_s = -1;
    __syncthreads();
    if (tid < QT) {
        int p = -1, row = 0, h = 0;
        if (tid < nq) {
            row = b * a.rps + r0 + tid / a.hp;
            h = hbase + tid % a.hp;
            p = a.row_pos[row];
        }
        qpos[tid] = p;
        qrow[tid] = row;
        qhead[tid] = h;
        mrun[tid] = -INFINITY;
        lrun[tid] = 0.f;
        if (p >= 0) atomicMax(&maxpos_s, p);
    }
    __syncthreads();
    // Spans past the group's last row position take no part (every workgroup of the group
    // derives the same live-span count from the row positions, and only live spans count in);
    // a group without any active row has its zero outputs written by span 0.
    const int nlive = maxpos_s >= 0 ? min(a.nsplit, maxpos_s / kSplit + 1) : 0;
    if (nlive == 0) {
        if (sp == 0)
            for (int idx = tid; idx < nq * HD; idx += kAttnT) {
                const int qi = idx / HD, d = idx % HD;
                a.out[(size_t)qrow[qi] * a.H * HD + qhead[qi] * HD + d] = 0.f;
            }
        return;
    }
    if (sp >= nlive) return;
    const int p_lo = sp * kSplit;
    const int maxpos = min(maxpos_s, p_lo + kSplit - 1);  // last position this span scores
    for (int idx = tid; idx < nq * HD; idx += kAttnT) {
        int qi = idx / HD, d = idx % HD;
        qs[idx] = a.q[(size_t)qrow[qi] * a.q_stride + qhead[qi] * HD + d] * a.scale;
    }
    const size_t head_base = (((size_t)a.layer * a.max_batch + b) * a.Hkv + kvh) * a.cap * HD;
    const float* kg = a.kc + head_base;
    const float* vg = a.vc + head_base;

    // output accumulators: thread owns dims d = tid % HD of query vectors qi = tid / HD + j * (T / HD)
    constexpr int QSTEP = kAttnT / HD;
    constexpr int NACC = QT / QSTEP;
    float acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j) acc[j] = 0.f;
    const int od = tid % HD, oq0 = tid / HD;

    // K/V chunk prefetch: each thread moves CL*HD/T float4 pairs per chunk
    constexpr int F4 = kAttnCL * HD / 4 / kAttnT;
    f4_t pk[F4], pv[F4];
    const int nchunks = maxpos >= p_lo ? (maxpos - p_lo) / kAttnCL + 1 : 0;
    const float* kgs = kg + (size_t)p_lo * HD;
    const float* vgs = vg + (size_t)p_lo * HD;
    if (nchunks > 0) fetch_chunk<HD, F4>(pk, pv, kgs, vgs, 0, maxpos - p_lo, tid);
    for (int c = 0; c < nchunks; ++c) {
        __syncthreads();  // previous chunk fully consumed
#pragma unroll
        for (int i = 0; i < F4; ++i) {
            int e4 = tid + i * kAttnT;
            int j = (e4 * 4) / HD, d = (e4 * 4) % HD;
            float* kd = ks + j * (HD + 1) + d;
            kd[0] = pk[i][0]; kd[1] = pk[i][1]; kd[2] = pk[i][2]; kd[3] = pk[i][3];
            *(f4_t*)(vs + j * HD + d) = pv[i];
        }
        __syncthreads();
        if (c + 1 < nchunks) fetch_chunk<HD, F4>(pk, pv, kgs, vgs, c + 1, maxpos - p_lo, tid);
        const int j0 = p_lo + c * kAttnCL;
        // scores of every (query, key) pair of the chunk; 64 threads per query vector
        for (int idx = tid; idx < nq * kAttnCL; idx += kAttnT) {
            int qi = idx / kAttnCL, j = idx % kAttnCL;
            float s = -INFINITY;
            if (j0 + j <= qpos[qi]) {
                const float* qr = qs + qi * HD;
                const float* kr = ks + j * (HD + 1);
                float d0 = 0.f;
#pragma unroll 8
                for (int d = 0; d < HD; ++d) d0 += qr[d] * kr[d];
                s = d0;
            }
            // row max and sum over the 64 keys held by this wave's 64 lanes
            float mx = at_wmax(s);
            float mnew = fmaxf(mrun[qi], mx);
            float p = (s == -INFINITY) ? 0.f : expf(s - mnew);
            float sum = at_wsum(p);
            ps[qi * kAttnCL + j] = p;
            if (j == 0) {
                float sc = mrun[qi] == -INFINITY ? 0.f : expf(mrun[qi] - mnew);
                rescale[qi] = sc;
                lrun[qi] = lrun[qi] * sc + sum;
                mrun[qi] = mnew;
            }
        }
        __syncthreads();
#pragma unroll
        for (int jj = 0; jj < NACC; ++jj) {
            int qi = oq0 + jj * QSTEP;
            if (qi < nq) {
                float o = acc[jj] * rescale[qi];
                const float* pr = ps + qi * kAttnCL;
#pragma unroll 8
                for (int j = 0; j < kAttnCL; ++j) o += pr[j] * vs[j * HD + od];
                acc[jj] = o;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int jj = 0; jj < NACC; ++jj) {
        int qi = oq0 + jj * QSTEP;
        if (qi < nq) {
            float* pp = a.part + (((size_t)qrow[qi] * a.H + qhead[qi]) * a.nsplit + sp) * (HD + 2);
            store_through(pp + od, acc[jj]);
            if (od == 0) {
                store_through(pp + HD, mrun[qi]);
                store_through(pp + HD + 1, lrun[qi]);
            }
        }
    }
    // the last live span of these query vectors to finish merges them in span order
    if (!arrive_last(a.cnt + wg, nlive, &last_flag)) return;
    for (int idx = tid; idx < nq * HD; idx += kAttnT) {
        int qi = idx / HD, d = idx % HD;
        int pos = qpos[qi];
        float res = 0.f;
        if (pos >= 0) {
            const float* pp = a.part + ((size_t)qrow[qi] * a.H + qhead[qi]) * a.nsplit * (HD + 2);
            // batches of 16 spans, every load of a batch issued before any is used (loads past
            // nlive re-read the last live span and are not added; a load behind a "live" test
            // would cost one memory round trip each), folded into a running maximum and sums
            float M = -INFINITY, L = 0.f, O = 0.f;
            for (int s0 = 0; s0 < nlive; s0 += 16) {
                float mv[16], lv[16], ov[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float* e = pp + (size_t)min(s0 + i, nlive - 1) * (HD + 2);
                    mv[i] = e[HD];
                    lv[i] = e[HD + 1];
                    ov[i] = e[d];
                }
                float Mn = M;
#pragma unroll
                for (int i = 0; i < 16; ++i) Mn = s0 + i < nlive ? fmaxf(Mn, mv[i]) : Mn;
                const float sc = M == -INFINITY ? 0.f : expf(M - Mn);
                L *= sc;
                O *= sc;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const bool live = s0 + i < nlive && mv[i] != -INFINITY;
                    const float w = live ? expf(mv[i] - Mn) : 0.f;
                    L += w * lv[i];
                    O += w * ov[i];
                }
                M = Mn;
            }
            res = L > 0.f ? O / L : 0.f;
        }
        a.out[(size_t)qrow[qi] * a.H * HD + qhead[qi] * HD + d] = res;
    }
}

// ---------------------------------------------------------------------------------------------
// Blocks of many rows per sequence (verify passes of 8 or more rows, prefill chunks, the
// training-objective forward): causal flash attention on fp32 matrix cores.  A workgroup owns
// 16 consecutive query rows of one sequence, one KV head and one span of key tiles; each of its
// 4 waves takes the query heads wave, wave + 4, ... of that KV head.  Per 16-position key tile,
// K and V are staged in LDS once for all the group's heads (the next tile is requested into
// registers while the current one is used).  A wave computes the transposed products, with
// v_mfma_f32_16x16x4_f32 (fp32 operands keep the cache's precision):
//   S^T = K Q^T   (16 keys x 16 queries; the head dimension walked as dim = g * HD/4 + s for
//                  lane group g and step s, so a lane's K operands are HD/4 adjacent floats)
//   O^T += V^T P^T (HD/16 tiles; output dim = i * HD/16 + t for tile row i and tile t, so a
//                  lane's V operands are HD/16 adjacent floats per key)
// In the result layout of S^T a lane holds four keys of one query (its column), which is also
// the layout P^T needs as an operand and the layout of that query's O^T rows: the online softmax
// runs in registers, with its max and sum taken over the four lane groups of a column by two
// lane-swap steps, and P never goes through LDS.  With few (sequence, KV head, row block)
// groups the keys are split into at most 16 spans of span_t tiles (about eight workgroups per
// compute unit): every span writes an un-normalised partial into k_attn's partial buffer and
// the last span of a group to arrive merges them in span order, all spans' loads at once.
// ---------------------------------------------------------------------------------------------
constexpr int kPaQ = 16;                  // query rows per workgroup
constexpr int kPaK = 16;                  // key positions per tile
constexpr int kPaMaxSpans = 16;           // spans per group (one merge batch)
constexpr int kPaMinRows = 8;             // rows per sequence from which blocks take k_pattn
typedef float pf4 __attribute__((ext_vector_type(4)));
typedef float pf2 __attribute__((ext_vector_type(2)));

// Max and sum over the four 16-lane groups of a wave (lanes l, l^16, l^32, l^48 hold one column).
__device__ __forceinline__ float pa_colmax(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float pa_colsum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// The last span of a (sequence, KV head, row block) group to finish merges the live spans in
// span order: a thread per (row, head, 4 dimensions), every span's (max, sum) and output
// requested at once.  qpos holds the block's row positions (-1: no row).
template <int HD>
__device__ void pa_span_merge(const AttnArgs& a, int grp_id, int nspan, int span_t, int ntile_all, int b, int kvh,
                              int i0, const int* qpos, int* last_flag) {
    if (!arrive_last(a.cnt + grp_id, nspan, last_flag)) return;
    const int tid = threadIdx.x, G = a.H / a.Hkv;
    const int nlive = min(nspan, ntile_all > 0 ? (ntile_all - 1) / span_t + 1 : 0);
    constexpr int D4 = HD / 4;
    for (int idx = tid; idx < kPaQ * G * D4; idx += 256) {
        const int i = idx / (G * D4), hh = (idx / D4) % G, d = (idx % D4) * 4;
        const int row = i0 + i;
        if (row >= a.rps) continue;
        const size_t orow = (size_t)(b * a.rps + row);
        const int h = kvh * G + hh;
        float4 res = make_float4(0.f, 0.f, 0.f, 0.f);
        if (qpos[i] >= 0 && nlive > 0) {
            const float* pp = a.part + (orow * a.H + h) * a.nsplit * (HD + 2);
            float m2[kPaMaxSpans], l2[kPaMaxSpans];
            float4 o2[kPaMaxSpans];
#pragma unroll
            for (int s2 = 0; s2 < kPaMaxSpans; ++s2) {
                const float* e2 = pp + (size_t)min(s2, nlive - 1) * (HD + 2);
                m2[s2] = e2[HD];
                l2[s2] = e2[HD + 1];
                o2[s2] = make_float4(e2[d], e2[d + 1], e2[d + 2], e2[d + 3]);
            }
            float M = -INFINITY;
#pragma unroll
            for (int s2 = 0; s2 < kPaMaxSpans; ++s2) M = s2 < nlive ? fmaxf(M, m2[s2]) : M;
            float L = 0.f;
#pragma unroll
            for (int s2 = 0; s2 < kPaMaxSpans; ++s2) {
                const float w = (s2 < nlive && m2[s2] != -INFINITY) ? expf(m2[s2] - M) : 0.f;
                L += w * l2[s2];
                res.x += w * o2[s2].x;
                res.y += w * o2[s2].y;
                res.z += w * o2[s2].z;
                res.w += w * o2[s2].w;
            }
            const float inv = L > 0.f ? 1.f / L : 0.f;
            res = make_float4(res.x * inv, res.y * inv, res.z * inv, res.w * inv);
        }
        *(float4*)(a.out + orow * a.H * HD + h * HD + d) = res;
    }
}

template <int HD>
__global__ __launch_bounds__(256) void k_pattn(AttnArgs a, int nspan, int span_t) {
    constexpr int KL = HD + 4;                            // padded LDS row of K and V
    constexpr int F4 = (kPaK * HD / 4 + 255) / 256;       // float4 of a K (or V) tile per thread
    constexpr int QD = HD / 4;                            // head dims per lane group in S^T
    constexpr int VD = HD / 16;                           // output dims per lane and key in O^T
    static_assert(QD % 4 == 0 && (VD % 4 == 0 || VD == 2), "head dim");
    __shared__ __attribute__((aligned(16))) float ks[kPaK * KL];
    __shared__ __attribute__((aligned(16))) float vs[kPaK * KL];
    __shared__ __attribute__((aligned(16))) float ot[4 * kPaQ * KL];  // per wave: O rows of one head
    __shared__ int qpos[kPaQ];
    __shared__ int maxpos_s;
    __shared__ int last_flag;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = a.H / a.Hkv;
    const int nqb = (a.rps + kPaQ - 1) / kPaQ;
    const int grp_id = blockIdx.x / nspan, sp = blockIdx.x % nspan;
    const int qb = grp_id % nqb;
    const int kvh = (grp_id / nqb) % a.Hkv;
    const int b = grp_id / (nqb * a.Hkv);
    const int i0 = qb * kPaQ;
    if (tid == 0) maxpos_s = -1;
    __syncthreads();
    if (tid < kPaQ) {
        int p = -1;
        if (i0 + tid < a.rps) p = a.row_pos[b * a.rps + i0 + tid];
        qpos[tid] = p;
        if (p >= 0) atomicMax(&maxpos_s, p);
    }
    __syncthreads();
    const int maxpos = maxpos_s;
    const int ntile_all = maxpos >= 0 ? maxpos / kPaK + 1 : 0;
    // this workgroup's key tiles: all of them, or one span
    const int t0 = nspan == 1 ? 0 : sp * span_t;
    const int t1 = nspan == 1 ? ntile_all : min(ntile_all, t0 + span_t);
    const size_t kvoff = (((size_t)a.layer * a.max_batch + b) * a.Hkv + kvh) * (size_t)a.cap * HD;
    const float* kg = a.kc + kvoff;
    const float* vg = a.vc + kvoff;
    const int col = lane & 15, grp = lane >> 4;  // MFMA layouts: column / row-group of this lane
    const int myq = qpos[col];                    // position of this lane's query row (-1: none)
    auto fetch = [&](int kt, float4 (&pk)[F4], float4 (&pv)[F4]) {
#pragma unroll
        for (int i = 0; i < F4; ++i) {
            const int e4 = tid + 256 * i;
            const int j = (e4 * 4) / HD, d = (e4 * 4) % HD, pos = kt * kPaK + j;
            pk[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            pv[i] = pk[i];
            if (e4 < kPaK * HD / 4 && pos <= maxpos) {
                pk[i] = *(const float4*)(kg + (size_t)pos * HD + d);
                pv[i] = *(const float4*)(vg + (size_t)pos * HD + d);
            }
        }
    };
    for (int hp = 0; hp * 4 < G; ++hp) {
        const int hh = hp * 4 + wave;
        const bool active = hh < G && t0 < t1;
        const int h = kvh * G + (hh < G ? hh : 0);
        // Q as the B operand of S^T: lane holds Q[row col][grp * QD + s], pre-scaled (rows past
        // the block re-read row 0 and are zeroed by the scale: no load depends on a branch,
        // which would cost one memory round trip per load)
        float qf[QD];
        {
            const int qrow = i0 + col;
            const bool ok = qrow < a.rps;
            const float* qp = a.q + (size_t)(b * a.rps + (ok ? qrow : 0)) * a.q_stride + h * HD + grp * QD;
            const float qs = ok ? a.scale : 0.f;
#pragma unroll
            for (int s = 0; s < QD; s += 4) {
                const pf4 x = *(const pf4*)(qp + s) * qs;
                qf[s] = x[0]; qf[s + 1] = x[1]; qf[s + 2] = x[2]; qf[s + 3] = x[3];
            }
        }
        pf4 o[VD];  // o[t][r] = O[query col][(4 grp + r) * VD + t]
#pragma unroll
        for (int t = 0; t < VD; ++t) o[t] = pf4{0.f, 0.f, 0.f, 0.f};
        float m_run = -INFINITY, l_run = 0.f;
        float4 pk[F4], pv[F4];
        if (t0 < t1) fetch(t0, pk, pv);
        for (int kt = t0; kt < t1; ++kt) {
            // stage this tile's K and V rows (positions past maxpos are zeros), request the next
            __syncthreads();
#pragma unroll
            for (int i = 0; i < F4; ++i) {
                const int e4 = tid + 256 * i;
                if (e4 < kPaK * HD / 4) {
                    const int j = (e4 * 4) / HD, d = (e4 * 4) % HD;
                    *(float4*)(ks + j * KL + d) = pk[i];
                    *(float4*)(vs + j * KL + d) = pv[i];
                }
            }
            __syncthreads();
            if (kt + 1 < t1) fetch(kt + 1, pk, pv);
            if (!active) continue;
            // operands from LDS, all requested before the first product: K[key col][grp*QD + s]
            // and V[key 4 grp + r][col * VD + t]
            float kf[QD], vf[4][VD];
#pragma unroll
            for (int s = 0; s < QD; s += 4) {
                const pf4 x = *(const pf4*)(ks + col * KL + grp * QD + s);
                kf[s] = x[0]; kf[s + 1] = x[1]; kf[s + 2] = x[2]; kf[s + 3] = x[3];
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float* vr = vs + (4 * grp + r) * KL + col * VD;
                if constexpr (VD == 2) {
                    const pf2 x = *(const pf2*)vr;
                    vf[r][0] = x[0]; vf[r][1] = x[1];
                } else {
#pragma unroll
                    for (int t = 0; t < VD; t += 4) {
                        const pf4 x = *(const pf4*)(vr + t);
                        vf[r][t] = x[0]; vf[r][t + 1] = x[1]; vf[r][t + 2] = x[2]; vf[r][t + 3] = x[3];
                    }
                }
            }
            // S^T = K Q^T in four independent accumulation chains; this lane then holds
            // S[query col][key 4 grp + r]
            pf4 sc4[4];
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) sc4[c4] = pf4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < QD; ++s)
                sc4[s & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf[s], qf[s], sc4[s & 3], 0, 0, 0);
            const pf4 sc = (sc4[0] + sc4[1]) + (sc4[2] + sc4[3]);
            // online softmax of query col over this tile's 16 keys
            const int kb = kt * kPaK + 4 * grp;
            float sv[4], mx = -INFINITY;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sv[r] = (myq >= 0 && kb + r <= myq) ? sc[r] : -INFINITY;
                mx = fmaxf(mx, sv[r]);
            }
            mx = pa_colmax(mx);
            const float mnew = fmaxf(m_run, mx);
            float pr[4], sum = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                pr[r] = sv[r] == -INFINITY ? 0.f : expf(sv[r] - mnew);
                sum += pr[r];
            }
            sum = pa_colsum(sum);
            const float scl = m_run == -INFINITY ? 0.f : expf(m_run - mnew);
            l_run = l_run * scl + sum;
            m_run = mnew;
#pragma unroll
            for (int t = 0; t < VD; ++t) o[t] *= scl;
            // O^T += V^T P^T: step r pairs key 4 grp + r with this lane's k slot
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int t = 0; t < VD; ++t)
                    o[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf[r][t], pr[r], o[t], 0, 0, 0);
        }
        // O through LDS into row-major order, then whole rows stored by the wave (a lane's own
        // values belong to one row: stored directly, each store would touch 16 rows)
        if (hh < G) {
            float* ow = ot + wave * (kPaQ * KL);
            const float inv = nspan == 1 ? ((myq >= 0 && l_run > 0.f) ? 1.f / l_run : 0.f) : 1.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float* dst = ow + col * KL + (4 * grp + r) * VD;
                if constexpr (VD == 2) {
                    *(pf2*)dst = pf2{o[0][r] * inv, o[1][r] * inv};
                } else {
#pragma unroll
                    for (int t = 0; t < VD; t += 4)
                        *(pf4*)(dst + t) = pf4{o[t][r] * inv, o[t + 1][r] * inv, o[t + 2][r] * inv, o[t + 3][r] * inv};
                }
            }
            if (nspan > 1 && grp == 0 && i0 + col < a.rps) {
                // this span's max and sum of the lane's row
                float* pp = a.part + (((size_t)(b * a.rps + i0 + col) * a.H + h) * a.nsplit + sp) * (HD + 2);
                store_through(pp + HD, m_run);
                store_through(pp + HD + 1, l_run);
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's rows are in LDS
            __builtin_amdgcn_wave_barrier();
            constexpr int RW = (HD + 63) / 64;  // values of one row per lane
            float rv[kPaQ][RW];                   // every row read before any is stored
#pragma unroll
            for (int i = 0; i < kPaQ; ++i)
#pragma unroll
                for (int j = 0; j < RW; ++j) rv[i][j] = ow[i * KL + min(lane + 64 * j, HD - 1)];
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int i = 0; i < kPaQ; ++i) {
                const size_t orow = (size_t)(b * a.rps + i0 + i);
#pragma unroll
                for (int j = 0; j < RW; ++j) {
                    const int d = lane + 64 * j;
                    if (i0 + i < a.rps && d < HD) {
                        if (nspan == 1) a.out[orow * a.H * HD + h * HD + d] = rv[i][j];
                        else store_through(a.part + ((orow * a.H + h) * a.nsplit + sp) * (HD + 2) + d, rv[i][j]);
                    }
                }
            }
        }
    }
    if (nspan == 1) return;
    pa_span_merge<HD>(a, grp_id, nspan, span_t, ntile_all, b, kvh, i0, qpos, &last_flag);
}

// Verify blocks of exactly 8 rows per sequence (k = 7), 4n query heads per KV head: two heads
// of 8 rows fill the 16 query columns of one S^T tile, so a key tile costs half the matrix work
// of the one-head layout (whose columns 8-15 would be empty).  Waves 0 and 1 take head pairs
// (0, 1) and (2, 3) of each pass of four heads over the even key tiles of the span, waves 2 and
// 3 the same pairs over the odd tiles; two tiles are staged per barrier pair.  The odd-tile wave
// of a pair hands its running max, sum and output to the even-tile wave through LDS (same lane
// layout), which merges them and stores the rows.  Arithmetic per product as in k_pattn.
template <int HD>
__global__ __launch_bounds__(256) void k_pattn_pk(AttnArgs a, int nspan, int span_t) {
    constexpr int KL = HD + 4;
    constexpr int F4 = (kPaK * HD / 4 + 255) / 256;
    constexpr int QD = HD / 4;
    constexpr int VD = HD / 16;
    static_assert(QD % 4 == 0 && (VD % 4 == 0 || VD == 2), "head dim");
    __shared__ __attribute__((aligned(16))) float ks[2][kPaK * KL];
    __shared__ __attribute__((aligned(16))) float vs[2][kPaK * KL];
    __shared__ __attribute__((aligned(16))) float ot[2 * kPaQ * KL];  // per head pair: hand-off, then O rows
    __shared__ float mlh[2][2][64];                                    // per head pair: max, sum per lane
    __shared__ int qpos[kPaQ];
    __shared__ int maxpos_s;
    __shared__ int last_flag;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = a.H / a.Hkv;
    const int grp_id = blockIdx.x / nspan, sp = blockIdx.x % nspan;
    const int kvh = grp_id % a.Hkv;
    const int b = grp_id / a.Hkv;
    if (tid == 0) maxpos_s = -1;
    __syncthreads();
    if (tid < kPaQ) {
        int p = -1;
        if (tid < 8) p = a.row_pos[b * 8 + tid];
        qpos[tid] = p;
        if (p >= 0) atomicMax(&maxpos_s, p);
    }
    __syncthreads();
    const int maxpos = maxpos_s;
    const int ntile_all = maxpos >= 0 ? maxpos / kPaK + 1 : 0;
    const int t0 = nspan == 1 ? 0 : sp * span_t;
    const int t1 = nspan == 1 ? ntile_all : min(ntile_all, t0 + span_t);
    const size_t kvoff = (((size_t)a.layer * a.max_batch + b) * a.Hkv + kvh) * (size_t)a.cap * HD;
    const float* kg = a.kc + kvoff;
    const float* vg = a.vc + kvoff;
    const int col = lane & 15, grp = lane >> 4;
    const int pr = wave & 1, half = wave >> 1;  // head pair of the pass, key-tile parity
    const int myq = qpos[col & 7];              // column col: row col % 8 of head 2 pr + col / 8
    // tiles kt and kt + 1 (the second past t1: zeros)
    auto fetch = [&](int kt, float4 (&pk)[2][F4], float4 (&pv)[2][F4]) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < F4; ++i) {
                const int e4 = tid + 256 * i;
                const int j = (e4 * 4) / HD, d = (e4 * 4) % HD, pos = (kt + u) * kPaK + j;
                pk[u][i] = make_float4(0.f, 0.f, 0.f, 0.f);
                pv[u][i] = pk[u][i];
                if (e4 < kPaK * HD / 4 && kt + u < t1 && pos <= maxpos) {
                    pk[u][i] = *(const float4*)(kg + (size_t)pos * HD + d);
                    pv[u][i] = *(const float4*)(vg + (size_t)pos * HD + d);
                }
            }
    };
    for (int hp = 0; hp * 4 < G; ++hp) {
        const int hh = hp * 4 + 2 * pr + (col >> 3);  // this lane column's head within the group
        const int h = kvh * G + hh;
        float qf[QD];
        {
            const float* qp = a.q + (size_t)(b * 8 + (col & 7)) * a.q_stride + h * HD + grp * QD;
#pragma unroll
            for (int s = 0; s < QD; s += 4) {
                const pf4 x = *(const pf4*)(qp + s) * a.scale;
                qf[s] = x[0]; qf[s + 1] = x[1]; qf[s + 2] = x[2]; qf[s + 3] = x[3];
            }
        }
        pf4 o[VD];  // o[t][r] = O[column col][(4 grp + r) * VD + t]
#pragma unroll
        for (int t = 0; t < VD; ++t) o[t] = pf4{0.f, 0.f, 0.f, 0.f};
        float m_run = -INFINITY, l_run = 0.f;
        float4 pk[2][F4], pv[2][F4];
        if (t0 < t1) fetch(t0, pk, pv);
        for (int kt = t0; kt < t1; kt += 2) {
            __syncthreads();
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int i = 0; i < F4; ++i) {
                    const int e4 = tid + 256 * i;
                    if (e4 < kPaK * HD / 4) {
                        const int j = (e4 * 4) / HD, d = (e4 * 4) % HD;
                        *(float4*)(ks[u] + j * KL + d) = pk[u][i];
                        *(float4*)(vs[u] + j * KL + d) = pv[u][i];
                    }
                }
            __syncthreads();
            if (kt + 2 < t1) fetch(kt + 2, pk, pv);
            const int mt = kt + half;
            if (mt >= t1) continue;  // uniform per wave; the next barrier is at the loop top
            const float* kss = ks[half];
            const float* vss = vs[half];
            float kf[QD], vf[4][VD];
#pragma unroll
            for (int s = 0; s < QD; s += 4) {
                const pf4 x = *(const pf4*)(kss + col * KL + grp * QD + s);
                kf[s] = x[0]; kf[s + 1] = x[1]; kf[s + 2] = x[2]; kf[s + 3] = x[3];
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float* vr = vss + (4 * grp + r) * KL + col * VD;
                if constexpr (VD == 2) {
                    const pf2 x = *(const pf2*)vr;
                    vf[r][0] = x[0]; vf[r][1] = x[1];
                } else {
#pragma unroll
                    for (int t = 0; t < VD; t += 4) {
                        const pf4 x = *(const pf4*)(vr + t);
                        vf[r][t] = x[0]; vf[r][t + 1] = x[1]; vf[r][t + 2] = x[2]; vf[r][t + 3] = x[3];
                    }
                }
            }
            pf4 sc4[4];
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) sc4[c4] = pf4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < QD; ++s)
                sc4[s & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf[s], qf[s], sc4[s & 3], 0, 0, 0);
            const pf4 sc = (sc4[0] + sc4[1]) + (sc4[2] + sc4[3]);
            const int kb = mt * kPaK + 4 * grp;
            float sv[4], mx = -INFINITY;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sv[r] = (myq >= 0 && kb + r <= myq) ? sc[r] : -INFINITY;
                mx = fmaxf(mx, sv[r]);
            }
            mx = pa_colmax(mx);
            const float mnew = fmaxf(m_run, mx);
            float pw[4], sum = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                pw[r] = sv[r] == -INFINITY ? 0.f : expf(sv[r] - mnew);
                sum += pw[r];
            }
            sum = pa_colsum(sum);
            const float scl = m_run == -INFINITY ? 0.f : expf(m_run - mnew);
            l_run = l_run * scl + sum;
            m_run = mnew;
#pragma unroll
            for (int t = 0; t < VD; ++t) o[t] *= scl;
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int t = 0; t < VD; ++t)
                    o[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf[r][t], pw[r], o[t], 0, 0, 0);
        }
        // the odd-tile wave of each pair hands its state over (lane layout), the even-tile wave
        // merges it
        float* ow = ot + pr * (kPaQ * KL);
        __syncthreads();
        if (half == 1) {
#pragma unroll
            for (int t = 0; t < VD; ++t) *(pf4*)(ow + (t * 64 + lane) * 4) = o[t];
            mlh[pr][0][lane] = m_run;
            mlh[pr][1][lane] = l_run;
        }
        __syncthreads();
        if (half == 0) {
            const float m2 = mlh[pr][0][lane], l2 = mlh[pr][1][lane];
            const float M = fmaxf(m_run, m2);
            const float s1 = m_run == -INFINITY ? 0.f : expf(m_run - M);
            const float s2 = m2 == -INFINITY ? 0.f : expf(m2 - M);
#pragma unroll
            for (int t = 0; t < VD; ++t) o[t] = o[t] * s1 + *(const pf4*)(ow + (t * 64 + lane) * 4) * s2;
            l_run = l_run * s1 + l2 * s2;
            m_run = M;
            // O through LDS into row-major order (this wave's own hand-off area, already read)
            const float inv = nspan == 1 ? ((myq >= 0 && l_run > 0.f) ? 1.f / l_run : 0.f) : 1.f;
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the hand-off reads are done
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float* dst = ow + col * KL + (4 * grp + r) * VD;
                if constexpr (VD == 2) {
                    *(pf2*)dst = pf2{o[0][r] * inv, o[1][r] * inv};
                } else {
#pragma unroll
                    for (int t = 0; t < VD; t += 4)
                        *(pf4*)(dst + t) = pf4{o[t][r] * inv, o[t + 1][r] * inv, o[t + 2][r] * inv, o[t + 3][r] * inv};
                }
            }
            if (nspan > 1 && grp == 0) {
                float* pp = a.part + (((size_t)(b * 8 + (col & 7)) * a.H + h) * a.nsplit + sp) * (HD + 2);
                store_through(pp + HD, m_run);
                store_through(pp + HD + 1, l_run);
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);
            __builtin_amdgcn_wave_barrier();
            constexpr int RW = (HD + 63) / 64;
            float rv[kPaQ][RW];
#pragma unroll
            for (int c = 0; c < kPaQ; ++c)
#pragma unroll
                for (int j = 0; j < RW; ++j) rv[c][j] = ow[c * KL + min(lane + 64 * j, HD - 1)];
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int c = 0; c < kPaQ; ++c) {
                const size_t orow = (size_t)(b * 8 + (c & 7));
                const int hc = kvh * G + hp * 4 + 2 * pr + (c >> 3);
#pragma unroll
                for (int j = 0; j < RW; ++j) {
                    const int d = lane + 64 * j;
                    if (d < HD) {
                        if (nspan == 1) a.out[orow * a.H * HD + hc * HD + d] = rv[c][j];
                        else store_through(a.part + ((orow * a.H + hc) * a.nsplit + sp) * (HD + 2) + d, rv[c][j]);
                    }
                }
            }
        }
    }
    if (nspan == 1) return;
    pa_span_merge<HD>(a, grp_id, nspan, span_t, ntile_all, b, kvh, 0, qpos, &last_flag);
}

static void launch_pattn(Engine& e, hipStream_t s, const AttnArgs& a, int nseq) {
    // the kernel reads query rows and writes output rows as 16-byte vectors
    if (a.q_stride % 4 || ((uintptr_t)a.q & 15) || ((uintptr_t)a.out & 15)) {
        e.bad_launch = true;
        return;
    }
    const int nqb = (a.rps + kPaQ - 1) / kPaQ;
    const int groups = nseq * a.Hkv * nqb;
    // few groups: split the keys into spans for about 2048 workgroups, eight per compute unit,
    // since spans past a sequence's length exit at once (at most 16 spans, within the decode
    // kernel's partial buffer and counters)
    // blocks of exactly 8 rows with a multiple of 4 query heads per KV head: two heads per
    // matrix tile (k_pattn_pk), which walks its span's key tiles two at a time
    const bool packed = a.rps == 8 && (a.H / a.Hkv) % 4 == 0;
    int nspan = 1, span_t = 1;
    if (groups < 256 && (size_t)groups <= e.ws.attn_cnt_n) {
        const int tiles = (a.cap + kPaK - 1) / kPaK;
        // (the packed kernel does half the matrix work per tile and measured best at ~768
        // workgroups: 79.8 us with 6 spans against 86.9 with 15 at the batched verify shape)
        nspan = std::min(std::min(kPaMaxSpans, a.nsplit), std::max(1, (packed ? 768 : 2048) / groups));
        span_t = (tiles + nspan - 1) / nspan;
        if (packed) span_t += span_t & 1;
        nspan = (tiles + span_t - 1) / span_t;
    }
    dim3 grid(groups * nspan);
    ProfEntry* pe = prof_slot(&e, kProfAttn, 0.0);
    hipEvent_t ea = pe ? pe->a : nullptr, eb = pe ? pe->b : nullptr;
    if (packed) {
        switch (a.hd) {
            case 32: hipExtLaunchKernelGGL(k_pattn_pk<32>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
            case 64: hipExtLaunchKernelGGL(k_pattn_pk<64>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
            case 128: hipExtLaunchKernelGGL(k_pattn_pk<128>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
            default: e.bad_launch = true; pe = nullptr; break;
        }
        if (pe) prof_commit(&e);
        return;
    }
    switch (a.hd) {
        case 32: hipExtLaunchKernelGGL(k_pattn<32>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
        case 64: hipExtLaunchKernelGGL(k_pattn<64>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
        case 128: hipExtLaunchKernelGGL(k_pattn<128>, grid, dim3(256), 0, s, ea, eb, 0, a, nspan, span_t); break;
        default: e.bad_launch = true; pe = nullptr; break;
    }
    if (pe) prof_commit(&e);
}

static size_t attn_lds(int hd, int qt) {
    return sizeof(float) * ((size_t)qt * hd + (size_t)kAttnCL * (hd + 1) + (size_t)kAttnCL * hd + (size_t)qt * kAttnCL);
}

// Query heads per workgroup: all heads of a KV group, so that each K/V row is read once for all
// of them (rows are then tiled 32/G at a time); one head per workgroup only for groups wider
// than a tile.
int attn_heads_per_wg(int nseq, int rps, int H, int Hkv) {
    (void)nseq;
    (void)rps;
    const int G = H / Hkv;
    return G > kAttnQT ? 1 : G;
}

void launch_attn(Engine& e, hipStream_t s, ModelDev& m, int layer, int rows, int rps, const float* q, int q_stride) {
    const sd2_dims& dm = m.dm;
    AttnArgs a;
    a.q = q; a.q_stride = q_stride; a.kc = m.kc; a.vc = m.vc; a.out = e.ws.attn; a.row_pos = e.ws.row_pos;
    a.rps = rps; a.H = dm.n_heads; a.Hkv = dm.n_kv_heads; a.hd = m.hd; a.cap = e.cap; a.max_batch = e.cfg.max_batch;
    a.layer = layer;
    int nseq = rows / rps;
    int G = dm.n_heads / dm.n_kv_heads;
    a.hp = attn_heads_per_wg(nseq, rps, dm.n_heads, dm.n_kv_heads);
    int rows_per_tile = kAttnQT / a.hp;
    a.nrt = (rps + rows_per_tile - 1) / rows_per_tile;
    a.ngrp = nseq * dm.n_kv_heads * a.nrt;
    a.scale = 1.0f / sqrtf((float)m.hd);
    a.nsplit = attn_nsplit(e.cap);
    a.part = e.ws.attn_part;
    a.cnt = e.ws.attn_cnt;
    if (rps >= kPaMinRows) {
        // many rows per sequence: flash attention on the matrix cores
        launch_pattn(e, s, a, nseq);
        return;
    }
    int members = G / a.hp;
    a.nsplit = attn_nsplit(e.cap);
    a.part = e.ws.attn_part;
    a.cnt = e.ws.attn_cnt;
    int nblk = (a.ngrp + kXcds - 1) / kXcds * kXcds * members * a.nsplit;
    ProfEntry* pe = prof_slot(&e, kProfAttn, 0.0);
    hipEvent_t ea = pe ? pe->a : nullptr, eb = pe ? pe->b : nullptr;
    // eight query-vector slots where a group's rows and heads fit them (decode steps: one or two
    // rows of a KV group), which quarters the query and score buffers in LDS; the row tiling,
    // and so the group count, is the same as with 32 slots (one tile)
    const bool q8 = a.hp * rps <= 8;
    switch (m.hd * (q8 ? -1 : 1)) {
        case 32: hipExtLaunchKernelGGL((k_attn<32, kAttnQT>), dim3(nblk), dim3(kAttnT), attn_lds(32, kAttnQT), s, ea, eb, 0, a); break;
        case 64: hipExtLaunchKernelGGL((k_attn<64, kAttnQT>), dim3(nblk), dim3(kAttnT), attn_lds(64, kAttnQT), s, ea, eb, 0, a); break;
        case 128: hipExtLaunchKernelGGL((k_attn<128, kAttnQT>), dim3(nblk), dim3(kAttnT), attn_lds(128, kAttnQT), s, ea, eb, 0, a); break;
        case -32: hipExtLaunchKernelGGL((k_attn<32, 8>), dim3(nblk), dim3(kAttnT), attn_lds(32, 8), s, ea, eb, 0, a); break;
        case -64: hipExtLaunchKernelGGL((k_attn<64, 8>), dim3(nblk), dim3(kAttnT), attn_lds(64, 8), s, ea, eb, 0, a); break;
        case -128: hipExtLaunchKernelGGL((k_attn<128, 8>), dim3(nblk), dim3(kAttnT), attn_lds(128, 8), s, ea, eb, 0, a); break;
        default: e.bad_launch = true; pe = nullptr; break;
    }
    if (pe) prof_commit(&e);
}

// Workgroups of the split-free attention grid for a launch shape (arrival counters needed).
size_t attn_groups(int rows, int rps, int H, int Hkv) {
    int nseq = rows / rps, G = H / Hkv;
    int hp = attn_heads_per_wg(nseq, rps, H, Hkv);
    int rows_per_tile = kAttnQT / hp;
    int nrt = (rps + rows_per_tile - 1) / rows_per_tile;
    int ngrp = nseq * Hkv * nrt;
    return (size_t)(ngrp + kXcds - 1) / kXcds * kXcds * (G / hp);
}

int attn_nsplit(int cap) { return (cap + kSplit - 1) / kSplit; }

}  // namespace sd2
