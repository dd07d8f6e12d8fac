// Weight-streaming projection for bf16 weights and up to 16 activation rows per launch.
//
//   Y[m][n] (op)= sum_k W[n][k] * xn[m][k],   xn = x (optionally RMS-normalised and scaled by gamma)
//
// Workgroups are persistent: each stages the activation slice xn[:, k0:k0+KR) in LDS once,
// as a bf16 hi/lo pair (xn ~= hi + lo to ~16 significant bits), then walks a strided list of
// 16-row weight tiles.  Its NW waves split the K-range; every lane streams 16-byte fragments
// so that the four lanes sharing a weight row read one contiguous 128-byte segment, and the
// next tile's fragments are requested before the current tile is multiplied, so HBM traffic
// never waits on the MFMA/LDS work.  The contraction runs on v_mfma_f32_16x16x32_bf16 twice
// per fragment (hi and lo), i.e. fp32 activations against bf16 weights.  The NW partial tiles
// are summed in LDS.  Weights are read exactly once.
//
// When the activation slice of the whole K does not fit in LDS, K is cut into S ranges; each
// range writes a partial tile (write-through), and the last workgroup to finish a tile adds the
// S partials in range order and applies the epilogue (see arrive_last).
//
// Epilogues: plain store (optional output-row map), residual add (+ per-16-column sums of
// squares of the new residual, consumed by the next RMSNorm), SwiGLU on paired gate/up
// tiles, and Q|K|V with rotate-half RoPE and the append of K and V to the cache.
#include <hip/hip_ext.h>

#include "device_common.h"
#include "engine.h"

namespace sd2 {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

typedef float wf2_t __attribute__((ext_vector_type(2)));
typedef __bf16 wbf2_t __attribute__((ext_vector_type(2)));

// hi/lo bf16 split of two fp32 values, packed as two bf16 words each (element 0 in the low
// half): hi = x rounded to nearest even, lo = (x - hi) rounded likewise; one hardware packed
// conversion per word (integer rounding took about six VALU operations per value)
__device__ __forceinline__ void split_hilo(float x0, float x1, uint32_t& hi, uint32_t& lo) {
    const wf2_t v = {x0, x1};
    const wbf2_t h = __builtin_convertvector(v, wbf2_t);
    const wbf2_t l = __builtin_convertvector(v - __builtin_convertvector(h, wf2_t), wbf2_t);
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, l);
}

struct WsArgs {
    const float* X;
    int ldx;
    const int32_t* in_map;
    int M;     // rows in this launch (<= 16)
    int row0;  // first row (of X / Y / row plans) handled by this launch
    int K;
    const uint16_t* gamma;
    float eps;
    const float* ss;  // [rows][nss] partial sums of squares of X rows (norm input)
    int nss;
    const uint16_t* W[3];
    int seg_tiles[3];
    int nseg;
    int mode;
    int tiles;
    float* Y;
    int ldy;
    const int32_t* out_map;
    float* ss_out;
    int KR, S, Gt;  // K-range per workgroup, number of K ranges, workgroups per K range
    float* part;    // S > 1: [tiles][S][SUBS][256]
    int32_t* cnt;   // S > 1: arrival counter per tile
    // Q|K|V mode
    int H, Hkv, hd;
    const int32_t *row_pos, *row_seq;
    const float *rcos, *rsin;
    float *qout, *kc, *vc;
    int cap, max_batch, layer;
    // MLP steering: bias of the row's sequence (row_seq), added to up (SwiGLU) or to the output
    // (Add), or null
    const float* ubias;
    int ub_ld;
};

// Weight row streamed by lane column n of a tile (segment resolution and the Q|K|V pairing
// of rotate-half partners i and i + hd/2 inside one tile).
__device__ __forceinline__ const uint16_t* tile_row(const WsArgs& a, int tile, int sub, int n) {
    if (a.mode == kEpiSwiglu) return a.W[sub] + (size_t)(tile * 16 + n) * a.K;
    int seg = 0, lt = tile;
    while (seg + 1 < a.nseg && lt >= a.seg_tiles[seg]) { lt -= a.seg_tiles[seg]; ++seg; }
    int wrow;
    if (a.mode == kEpiQkv) {
        int per_head = a.hd / 16;
        int h = lt / per_head, j = lt % per_head;
        wrow = h * a.hd + (n < 8 ? 8 * j + n : a.hd / 2 + 8 * j + (n - 8));
    } else {
        wrow = lt * 16 + n;
    }
    return a.W[seg] + (size_t)wrow * a.K;
}

// Epilogue of one finished 16x16 tile; element (m, c) is held by thread t = 16m + c of the
// first 256 threads.  `v` holds the value per sub-tile.
template <int SUBS>
// Rows row0 .. row0 + nrows - 1 of the launch (at most 16).
__device__ __forceinline__ void tile_epilogue(const WsArgs& a, int tile, const float* v, int row0, int nrows) {
    const int tid = threadIdx.x;
    const int em = tid >> 4, ec = tid & 15;
    const bool valid = em < nrows;
    const int row = row0 + em;
    if (a.mode == kEpiStore) {
        if (valid) {
            int orow = a.out_map ? a.out_map[row] : row;
            if (orow >= 0) a.Y[(size_t)orow * a.ldy + tile * 16 + ec] = v[0];
        }
    } else if (a.mode == kEpiAdd) {
        float nv = 0.0f;
        if (valid) {
            float* yp = a.Y + (size_t)row * a.ldy + tile * 16 + ec;
            nv = *yp + v[0];
            if (a.ubias) nv += a.ubias[(size_t)a.row_seq[row] * a.ub_ld + tile * 16 + ec];
            *yp = nv;
        }
        float sq = nv * nv;
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 16);
        if (valid && ec == 0) a.ss_out[(size_t)row * a.tiles + tile] = sq;
    } else if (a.mode == kEpiSwiglu) {
        if (valid) {
            float up = v[SUBS - 1];
            if (a.ubias) up += a.ubias[(size_t)a.row_seq[row] * a.ub_ld + tile * 16 + ec];
            a.Y[(size_t)row * a.ldy + tile * 16 + ec] = silu(v[0]) * up;
        }
    } else {
        float partner = __shfl_xor(v[0], 8, 16);
        if (!valid) return;
        int seg = 0, lt = tile;
        while (seg + 1 < a.nseg && lt >= a.seg_tiles[seg]) { lt -= a.seg_tiles[seg]; ++seg; }
        int per_head = a.hd / 16;
        int h = lt / per_head, j = lt % per_head;
        int half = a.hd / 2;
        int i = 8 * j + (ec & 7);
        int dim = ec < 8 ? i : half + i;
        int pos = a.row_pos[row];
        float out = v[0];
        if (seg < 2) {
            int pp = pos < 0 ? 0 : pos;
            float c = a.rcos[(size_t)pp * half + i], sn = a.rsin[(size_t)pp * half + i];
            out = ec < 8 ? v[0] * c - partner * sn : v[0] * c + partner * sn;
        }
        if (seg == 0) {
            a.qout[(size_t)row * a.H * a.hd + h * a.hd + dim] = out;
        } else if (pos >= 0) {
            int b = a.row_seq[row];
            size_t idx = ((((size_t)a.layer * a.max_batch + b) * a.Hkv + h) * a.cap + pos) * a.hd + dim;
            if (seg == 1) a.kc[idx] = out;
            else a.vc[idx] = out;
        }
    }
}

// Sum of one row's slice sums of squares over a wave (lane l takes slices l, l + 64, ...): loads in
// batches of eight per lane with clamped indexes, so that none waits for the one before it.
// row < 0: 0.
__device__ __forceinline__ float row_sumsq(const float* ss, int nss, int row, int lane) {
    const float* rp = ss + (size_t)max(row, 0) * nss;
    float sm = 0.0f;
    for (int t0 = 0; t0 < nss; t0 += 512) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = rp[min(t0 + lane + 64 * u, nss - 1)];
#pragma unroll
        for (int u = 0; u < 8; ++u) sm += (row >= 0 && t0 + lane + 64 * u < nss) ? v[u] : 0.f;
    }
    return sm;
}

template <int NW, int STEPS, int SUBS>
__global__ __launch_bounds__(NW * 64) void k_wsgemv(WsArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ float inv_rms[16];
    __shared__ int src_row[16];
    __shared__ int last_flag;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int M = a.M;
    const int KR = a.KR;
    const int ldk = KR + 8;  // padded row stride (bf16 elements) of the LDS slices
    const int s = blockIdx.x % a.S;
    const int g = blockIdx.x / a.S;
    const int k0 = s * KR;
    uint16_t* xh = (uint16_t*)smem;
    uint16_t* xl = xh + (size_t)M * ldk;
    float* red = (float*)(xl + (size_t)M * ldk);  // [NW][256]

    const int n = lane & 15, q = lane >> 4;
    const int kw0 = wave * (KR / NW);

    // The workgroup's work is a sequence of sub-tiles u = 0, 1, ...: tile g + (u / SUBS) * Gt,
    // sub-tile u % SUBS (SwiGLU: gate then up).  Two sub-tiles of weight fragments are kept in
    // flight in two register buffers.
    const int ntile_mine = a.tiles > g ? (a.tiles - g + a.Gt - 1) / a.Gt : 0;
    const int nsub_mine = ntile_mine * SUBS;
    u32x4_t wa[STEPS][2], wb[STEPS][2];
    auto issue = [&](u32x4_t (&buf)[STEPS][2], int u) {
        const int tile = g + (u / SUBS) * a.Gt;
        const uint16_t* wp = tile_row(a, tile, u % SUBS, n) + k0 + kw0 + 16 * q;
#pragma unroll
        for (int st = 0; st < STEPS; ++st)
#pragma unroll
            for (int h = 0; h < 2; ++h) buf[st][h] = *(const u32x4_t*)(wp + st * 64 + 8 * h);
    };

    // ---- prologue.  Loads return in issue order, so the small activation loads go first, then
    //      the first weight sub-tile, then the RMSNorm statistics (needed only by the epilogue:
    //      the row scale 1/rms is applied to the outputs, the gain to the staged activations) ----
    if (tid < 16) {
        int src = -1;
        if (tid < M) src = a.in_map ? a.in_map[a.row0 + tid] : a.row0 + tid;
        src_row[tid] = src;
        inv_rms[tid] = 1.0f;
    }
    __syncthreads();
    constexpr int XB = 16;  // activation float4 loads per thread issued ahead of the weights
    const int n4 = KR / 4;
    const int nx = M * n4;  // float4 groups of the slice, row-major
    float4 xv[XB];
#pragma unroll
    for (int i = 0; i < XB; ++i) {
        const int idx = tid + i * NW * 64;
        if (idx < nx) {
            const int m = idx / n4, kk = (idx % n4) * 4;
            const int src = src_row[m];
            xv[i] = src >= 0 ? *(const float4*)(a.X + (size_t)src * a.ldx + k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    // the gain words of the same columns, all requested before any is used (a load under a
    // per-element test would wait for everything in flight, the weights included)
    uint2 gv[XB];
    if (a.gamma) {
#pragma unroll
        for (int i = 0; i < XB; ++i) {
            const int idx = min(tid + i * NW * 64, nx - 1);
            gv[i] = *(const uint2*)(a.gamma + k0 + (idx % n4) * 4);
        }
    } else {
#pragma unroll
        for (int i = 0; i < XB; ++i) gv[i] = make_uint2(0x3f803f80u, 0x3f803f80u);  // bf16 ones
    }
    if (nsub_mine > 0) issue(wa, 0);
    float ssum = 0.0f;
    const int ss_row = wave < M ? src_row[wave] : -1;
    if (a.gamma) ssum = row_sumsq(a.ss, a.nss, ss_row, lane);
    auto stage = [&](const float4& v, int idx, uint2 gw) {
        const int m = idx / n4, kk = (idx % n4) * 4;
        float gm[4] = {1.f, 1.f, 1.f, 1.f};
        if (a.gamma) {
            gm[0] = bf16_lo(gw.x); gm[1] = bf16_hi(gw.x); gm[2] = bf16_lo(gw.y); gm[3] = bf16_hi(gw.y);
        }
        uint32_t h0, h1, l0, l1;
        split_hilo(v.x * gm[0], v.y * gm[1], h0, l0);
        split_hilo(v.z * gm[2], v.w * gm[3], h1, l1);
        *(uint2*)(xh + (size_t)m * ldk + kk) = make_uint2(h0, h1);
        *(uint2*)(xl + (size_t)m * ldk + kk) = make_uint2(l0, l1);
    };
#pragma unroll
    for (int i = 0; i < XB; ++i) {
        const int idx = tid + i * NW * 64;
        if (idx < nx) stage(xv[i], idx, gv[i]);
    }
    // slices larger than XB float4 per thread (not used by the planned shapes) stage the rest here
    for (int idx = tid + XB * NW * 64; idx < nx; idx += NW * 64) {
        const int m = idx / n4, kk = (idx % n4) * 4;
        const int src = src_row[m];
        float4 v = src >= 0 ? *(const float4*)(a.X + (size_t)src * a.ldx + k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
        const uint2 gw = a.gamma ? *(const uint2*)(a.gamma + k0 + kk) : make_uint2(0x3f803f80u, 0x3f803f80u);
        stage(v, idx, gw);
    }
    if (nsub_mine > 1) issue(wb, 1);
    if (a.gamma) {
        ssum = wave_sum(ssum);
        if (lane == 0 && wave < M) inv_rms[wave] = rsqrtf(ssum / (float)a.K + a.eps);
        // rows beyond the number of waves (M > NW)
        for (int m = NW + wave; m < M; m += NW) {
            float sm = row_sumsq(a.ss, a.nss, src_row[m], lane);
            sm = wave_sum(sm);
            if (lane == 0) inv_rms[m] = rsqrtf(sm / (float)a.K + a.eps);
        }
    }
    __syncthreads();

    const bool arow = n < M;
    float stash = 0.0f;  // gate value of the current SwiGLU tile (threads < 256)
    auto compute = [&](u32x4_t (&buf)[STEPS][2], int u) {
        floatx4_t acc = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int kk = kw0 + st * 64 + 16 * q + 8 * h;
                bf16x8_t ah = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0}, al = ah;
                if (arow) {
                    ah = *(const bf16x8_t*)(xh + (size_t)n * ldk + kk);
                    al = *(const bf16x8_t*)(xl + (size_t)n * ldk + kk);
                }
                bf16x8_t b = __builtin_bit_cast(bf16x8_t, buf[st][h]);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b, acc, 0, 0, 0);
            }
        }
        // sum the NW waves' tiles: element (m, c) = (t / 16, t % 16); scale by the row's 1/rms
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave * 256 + (4 * q + i) * 16 + n] = acc[i];
        __syncthreads();
        const int tile = g + (u / SUBS) * a.Gt;
        const int sub = u % SUBS;
        float x = 0.0f;
        if (tid < 256) {
#pragma unroll
            for (int w = 0; w < NW; ++w) x += red[w * 256 + tid];
            x *= inv_rms[tid >> 4];
        }
        if (SUBS == 2 && sub == 0) {
            stash = x;
        } else if (a.S == 1) {
            float v[2] = {SUBS == 2 ? stash : x, x};
            if (tid < 256) tile_epilogue<SUBS>(a, tile, v, a.row0, a.M);
        } else {
            // K split over S workgroups: the last to finish this tile adds the partials in order
            float* pt = a.part + (size_t)tile * a.S * SUBS * 256;
            if (tid < 256) {
                store_through(pt + (size_t)s * SUBS * 256 + tid, SUBS == 2 ? stash : x);
                if (SUBS == 2) store_through(pt + (size_t)s * SUBS * 256 + 256 + tid, x);
            }
            if (arrive_last(a.cnt + tile, a.S, &last_flag) && tid < 256) {
                float p0[8], p1[8];
                float v[2] = {0.f, 0.f};
                for (int s0 = 0; s0 < a.S; s0 += 8) {
                    const int ns = min(8, a.S - s0);
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        if (i < ns) {
                            p0[i] = pt[(size_t)(s0 + i) * SUBS * 256 + tid];
                            if (SUBS == 2) p1[i] = pt[(size_t)(s0 + i) * SUBS * 256 + 256 + tid];
                        }
                    }
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        if (i < ns) {
                            v[0] += p0[i];
                            if (SUBS == 2) v[1] += p1[i];
                        }
                    }
                }
                if (SUBS == 1) v[1] = v[0];
                tile_epilogue<SUBS>(a, tile, v, a.row0, a.M);
            }
        }
        __syncthreads();
    };

    // ---- sub-tile loop: after a buffer is consumed it is refilled two sub-tiles ahead ----
    for (int u = 0; u < nsub_mine; u += 2) {
        compute(wa, u);
        if (u + 2 < nsub_mine) issue(wa, u + 2);
        if (u + 1 >= nsub_mine) break;
        compute(wb, u + 1);
        if (u + 3 < nsub_mine) issue(wb, u + 3);
    }
}

// ===========================================================================
// Many-row projections (prefill chunks, large batches, verify passes of more than 16 rows): an
// MFMA GEMM.  A workgroup computes 64 activation rows (4 groups of 16) against 8 weight sub-tiles
// of 16 rows (two per wave), walking K in steps of 128 columns through a two-deep pipeline: the
// activation slice of step i + 1 sits in the second of two LDS buffers (hi/lo bf16 planes, gain
// applied, as in k_wsgemv) and its weight fragments in a second register set while step i's
// MFMAs run, and the loads of step i + 2 are issued as soon as step i + 1's activations have been
// staged.  Every weight fragment meets all 4 row groups.  Epilogues are k_wsgemv's, per 16-row
// group.
// ===========================================================================
constexpr int kPgRows = 64;           // activation rows per workgroup
constexpr int kPgTW = 2;              // weight sub-tiles per wave
constexpr int kPgKC = 128;            // K columns per step
constexpr int kPgLdk = kPgKC + 8;     // padded LDS row stride (bf16 elements)
constexpr int kPgX4 = kPgRows * kPgKC / 4 / 256;  // float4 of a step's activation slice per thread
constexpr size_t kPgPlane = (size_t)kPgRows * kPgLdk;           // bf16 elements of one plane
constexpr size_t kPgLds = 2 * 2 * kPgPlane * 2;  // two buffers of hi and lo planes (also holds the 32 KB of results)
static_assert(kPgLds >= 4 * kPgTW * 4 * 256 * 4, "result staging must fit the activation planes");

// K ranges for a many-row projection: split while the grid stays within 2 workgroups per CU and
// every range keeps at least 1024 columns (a multiple of 256); 512 with a single 64-row block,
// whose grid is the smallest (the 32-row first drafter step of a 16-sequence batch).  Shared by
// the launch and the workspace sizing.
int pg_split(int M, int N, int K, int subs) {
    const int nt = 4 * kPgTW / subs;
    const int nblk_m = (M + kPgRows - 1) / kPgRows;
    const int nblk_n = (N / 16 + nt - 1) / nt;
    const int blocks = 8 * nblk_m * ((nblk_n + 7) / 8);
    int S = 1;
    const int min_range = nblk_m == 1 ? 512 : 1024;
    while (blocks * S * 2 <= 512 && (K / (S * 2)) % 256 == 0 && K / (S * 2) >= min_range && K % (S * 2) == 0) S *= 2;
    return S;
}

template <int SUBS>
__global__ __launch_bounds__(256, 2) void k_pgemm(WsArgs a, int nblk_m, int nbs) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ float inv_rms[kPgRows];
    __shared__ int src_row[kPgRows];
    constexpr int NT = 4 * kPgTW / SUBS;  // 16-row output tiles per workgroup
    __shared__ int last_tile[NT];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = lane & 15, q = lane >> 4;
    // block -> (n block, m block): workgroups are dealt to the 8 XCDs in turn, so blocks b, b + 8,
    // ... share an XCD; they take the m blocks of one n block, whose weights then come from that
    // XCD's L2 after the first read
    // K range s of a.S (blocks of one range are contiguous); within it, as for S = 1
    const int s = blockIdx.x / nbs;
    const int bb = blockIdx.x % nbs;
    const int xcd = bb & 7, r = bb >> 3;
    const int mb = r % nblk_m;
    const int nb = xcd + 8 * (r / nblk_m);
    const int tile0 = nb * NT;
    if (tile0 >= a.tiles) return;  // grid padding (uniform per workgroup)
    const int m0 = mb * kPgRows;
    const int M = a.M;
    if (tid < kPgRows) {
        const int row = m0 + tid;
        int src = -1;
        if (row < M) src = a.in_map ? a.in_map[row] : row;
        src_row[tid] = src;
        inv_rms[tid] = 1.0f;
    }
    __syncthreads();
    // this wave's sub-tiles: SwiGLU waves 0, 1 take gate rows and waves 2, 3 the up rows of the
    // same features; a tile past the end is read clamped and never written
    const int sub = SUBS == 2 ? wave >> 1 : 0;
    const uint16_t* wrow[kPgTW];
#pragma unroll
    for (int j = 0; j < kPgTW; ++j) {
        const int tile = tile0 + (SUBS == 2 ? (wave & 1) * kPgTW : wave * kPgTW) + j;
        wrow[j] = tile_row(a, min(tile, a.tiles - 1), sub, n) + 16 * q;
    }
    uint16_t* const planes = (uint16_t*)smem;  // [buffer][hi, lo][64][kPgLdk]
    floatx4_t acc[kPgTW][4];
#pragma unroll
    for (int j = 0; j < kPgTW; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[j][g] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    const int KS = a.K / a.S, kb = s * KS, nstep = KS / kPgKC;
    typedef u32x4_t WFrag[kPgTW][2][2];
    // weight fragments of step i: lane (n, q) holds row n of each sub-tile, columns
    // 64 st + 16 q + 8 h + [0, 8) of the step (A is read with the same column order)
    auto load_w = [&](int i, WFrag& w) {
        const int k0 = kb + i * kPgKC;
#pragma unroll
        for (int j = 0; j < kPgTW; ++j)
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int h = 0; h < 2; ++h) w[j][st][h] = *(const u32x4_t*)(wrow[j] + k0 + st * 64 + 8 * h);
    };
    // 64 rows x 128 columns of fp32 activations: kPgX4 float4 per thread, row-major (a thread's
    // float4 all sit at the same 4 columns, so it needs one word pair of the gain per step,
    // requested with them)
    const int kk_t = (tid & 31) * 4;
    auto load_x = [&](int i, float4 (&xv)[kPgX4], uint2& gw) {
        const int k0 = kb + i * kPgKC;
#pragma unroll
        for (int e = 0; e < kPgX4; ++e) {
            const int m = (tid + e * 256) >> 5;
            const int src = src_row[m];
            xv[e] = src >= 0 ? *(const float4*)(a.X + (size_t)src * a.ldx + k0 + kk_t) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        gw = a.gamma ? *(const uint2*)(a.gamma + k0 + kk_t) : make_uint2(0x3f803f80u, 0x3f803f80u);
    };
    // gain, then the hi/lo bf16 split of step i's slice into buffer (i & 1)
    auto stage = [&](int i, const float4 (&xv)[kPgX4], uint2 gw) {
        uint16_t* xh = planes + (size_t)(i & 1) * 2 * kPgPlane;
        uint16_t* xl = xh + kPgPlane;
        const float gm[4] = {bf16_lo(gw.x), bf16_hi(gw.x), bf16_lo(gw.y), bf16_hi(gw.y)};
#pragma unroll
        for (int e = 0; e < kPgX4; ++e) {
            const int m = (tid + e * 256) >> 5, kk = kk_t;
            uint32_t h0, h1, l0, l1;
            split_hilo(xv[e].x * gm[0], xv[e].y * gm[1], h0, l0);
            split_hilo(xv[e].z * gm[2], xv[e].w * gm[3], h1, l1);
            *(uint2*)(xh + m * kPgLdk + kk) = make_uint2(h0, h1);
            *(uint2*)(xl + m * kPgLdk + kk) = make_uint2(l0, l1);
        }
    };
    auto mma = [&](int i, const WFrag& w) {
        const uint16_t* xh = planes + (size_t)(i & 1) * 2 * kPgPlane;
        const uint16_t* xl = xh + kPgPlane;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int kk = st * 64 + 16 * q + 8 * h;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const bf16x8_t ah = *(const bf16x8_t*)(xh + (g * 16 + n) * kPgLdk + kk);
                    const bf16x8_t al = *(const bf16x8_t*)(xl + (g * 16 + n) * kPgLdk + kk);
#pragma unroll
                    for (int j = 0; j < kPgTW; ++j) {
                        const bf16x8_t b = __builtin_bit_cast(bf16x8_t, w[j][st][h]);
                        acc[j][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b, acc[j][g], 0, 0, 0);
                        acc[j][g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b, acc[j][g], 0, 0, 0);
                    }
                }
            }
        }
    };
    // Pipeline: step i's MFMAs (weights wa for even i, wb for odd), then step i + 1's activations
    // staged into the other buffer, then the loads of step i + 2 into the registers just freed;
    // one barrier per step (a buffer is rewritten only after every wave has passed the barrier
    // that follows its last read).
    WFrag wa, wb;
    float4 xv[kPgX4];
    uint2 gw;
    load_x(0, xv, gw);
    load_w(0, wa);
    // RMSNorm statistics (used by the epilogue only), requested behind the first step's loads:
    // four threads per row, each summing every fourth float4 of the row's partial sums of squares
    if (a.gamma) {
        const int m = tid >> 2, p = tid & 3;
        const int src = src_row[m];
        float sm = 0.0f;
        // eight float4 per thread in flight at once, indexes clamped and the extra ones dropped
        // (loads under a loop test would each wait for the previous one)
        const float4* sp = (const float4*)(a.ss + (size_t)max(src, 0) * a.nss);
        const int n4s = a.nss / 4;
        for (int f0 = 0; f0 < n4s; f0 += 32) {
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = sp[min(f0 + p + 4 * u, n4s - 1)];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                sm += (src >= 0 && f0 + p + 4 * u < n4s) ? (v[u].x + v[u].y) + (v[u].z + v[u].w) : 0.f;
        }
        sm += __shfl_xor(sm, 1, 4);
        sm += __shfl_xor(sm, 2, 4);
        if (p == 0) inv_rms[m] = rsqrtf(sm / (float)a.K + a.eps);
    }
    stage(0, xv, gw);
    if (nstep > 1) {
        load_x(1, xv, gw);
        load_w(1, wb);
    }
    __syncthreads();
    for (int i = 0; i < nstep; i += 2) {
        mma(i, wa);
        if (i + 1 < nstep) stage(i + 1, xv, gw);
        if (i + 2 < nstep) {
            load_x(i + 2, xv, gw);
            load_w(i + 2, wa);
        }
        __syncthreads();
        if (i + 1 >= nstep) break;
        mma(i + 1, wb);
        if (i + 2 < nstep) stage(i + 2, xv, gw);
        if (i + 3 < nstep) {
            load_x(i + 3, xv, gw);
            load_w(i + 3, wb);
        }
        __syncthreads();
    }
    __syncthreads();  // planes free: results go to LDS, slot (wave * TW + j, group g)
    float* red = (float*)smem;
#pragma unroll
    for (int j = 0; j < kPgTW; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[((wave * kPgTW + j) * 4 + g) * 256 + (4 * q + i) * 16 + n] = acc[j][g][i];
    __syncthreads();
    // per output tile and row group: element (m, c) at thread 16 m + c; SwiGLU's up value of
    // local tile lt sits 2 TW slots after its gate value.  With K ranges, each range stores its
    // sums of every (tile, m block) it holds, waits once for all of those stores, and counts in on
    // all of its tiles at once; the last range to arrive at a tile adds the S partials in range
    // order.
    if (a.S > 1) {
        for (int lt = 0; lt < NT; ++lt) {
            const int tile = tile0 + lt;
            if (tile >= a.tiles) break;
            float* pt = a.part + (size_t)(tile * nblk_m + mb) * a.S * SUBS * 1024;
#pragma unroll
            for (int sub = 0; sub < SUBS; ++sub)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    store_through(pt + ((size_t)s * SUBS + sub) * 1024 + g * 256 + tid,
                                  red[((lt + sub * 2 * kPgTW) * 4 + g) * 256 + tid]);
        }
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores have completed
        __syncthreads();
        if (tid < NT) {
            const int tile = tile0 + tid;
            int last = 0;
            if (tile < a.tiles) {
                int32_t* c = a.cnt + tile * nblk_m + mb;
                const int prev = __hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                last = prev == a.S - 1;
                if (last) __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            last_tile[tid] = last;
        }
        __syncthreads();
    }
    for (int lt = 0; lt < NT; ++lt) {
        const int tile = tile0 + lt;
        if (tile >= a.tiles) break;
        if (a.S > 1 && !last_tile[lt]) continue;
        float sum[4][SUBS];
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int sub = 0; sub < SUBS; ++sub) sum[g][sub] = red[((lt + sub * 2 * kPgTW) * 4 + g) * 256 + tid];
        if (a.S > 1) {
            // the S ranges' partials of all 4 row groups, 8 ranges per round trip (loads past S
            // re-read the last range and are not added)
            const float* pt = a.part + (size_t)(tile * nblk_m + mb) * a.S * SUBS * 1024 + tid;
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int sub = 0; sub < SUBS; ++sub) sum[g][sub] = 0.f;
            for (int s0 = 0; s0 < a.S; s0 += 8) {
                float p[8][4][SUBS];
#pragma unroll
                for (int r = 0; r < 8; ++r)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
#pragma unroll
                        for (int sub = 0; sub < SUBS; ++sub)
                            p[r][g][sub] = pt[((size_t)min(s0 + r, a.S - 1) * SUBS + sub) * 1024 + g * 256];
#pragma unroll
                for (int r = 0; r < 8; ++r)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
#pragma unroll
                        for (int sub = 0; sub < SUBS; ++sub) sum[g][sub] += s0 + r < a.S ? p[r][g][sub] : 0.f;
            }
        }
        for (int g = 0; g < 4; ++g) {
            const int row0 = m0 + g * 16;
            if (row0 >= M) break;
            const float sc = inv_rms[g * 16 + (tid >> 4)];
            float v[2];
            v[0] = sum[g][0] * sc;
            v[1] = SUBS == 2 ? sum[g][SUBS - 1] * sc : v[0];
            tile_epilogue<SUBS>(a, tile, v, row0, min(16, M - row0));
        }
    }
}

hipError_t wsgemv_setup() {
    hipError_t e1 = hipFuncSetAttribute((const void*)k_pgemm<1>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kPgLds);
    hipError_t e2 = hipFuncSetAttribute((const void*)k_pgemm<2>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kPgLds);
    return e1 != hipSuccess ? e1 : e2;
}

constexpr int kLdsBudget = 160 * 1024 - 2048;
// Activation bytes a workgroup stages: K is split until each workgroup's slice of the rows fits
// this (16 rows of 2048 columns would be 128 KB read from L2 by every workgroup for one 64 KB
// weight tile, at one workgroup per CU); without such a split, the smallest that fits LDS.
constexpr size_t kWsStageMax = 64 * 1024;

static size_t lds_bytes(int rows, int KR, int NW) {
    return (size_t)rows * (KR + 8) * 2 * 2 + (size_t)NW * 256 * 4;
}

// Plan: number of K ranges S (1 when the whole activation row fits in LDS), K-range KR,
// waves NW and fragment steps per lane, and how many workgroups walk the tiles.
WsPlan ws_plan(int M, int N, int K, int mode) {
    WsPlan p{};
    int rows = M < 16 ? M : 16;
    (void)mode;
    p.tiles = N / 16;
    // first pass: the smallest split whose staged slice fits kWsStageMax; second: any that fits
    for (int pass = 0; pass < 2 && !p.S; ++pass)
    for (int S = 1; S <= K / 256; ++S) {
        if (K % S) continue;
        int KR = K / S;
        if (KR % 256) continue;
        if (pass == 0 && (size_t)rows * KR * 4 > kWsStageMax) continue;
        // waves: each a multiple of 64 columns; two fragment buffers of 8*steps VGPRs each must
        // leave room in the 512-entry register file (8 steps with <= 8 waves, 4 with 16 waves)
        int NW = 0, steps = 0;
        for (int nw = 4; nw <= 16; nw *= 2) {
            if (KR % (nw * 64)) continue;
            int st = KR / (nw * 64);
            if (st > (nw == 16 ? 4 : 8)) continue;
            NW = nw;
            steps = st;
            break;
        }
        if (!NW) continue;
        if (lds_bytes(rows, KR, NW) > (size_t)kLdsBudget) continue;
        p.S = S;
        p.KR = KR;
        p.NW = NW;
        p.steps = steps;
        break;
    }
    if (!p.S) return p;
    size_t lds = lds_bytes(rows, p.KR, p.NW);
    int per_cu = (int)((160 * 1024) / (lds + 1024));
    if (per_cu < 1) per_cu = 1;
    if (per_cu > 2) per_cu = 2;
    int want = 256 * per_cu;
    int gt = want / p.S;
    if (gt < 1) gt = 1;
    if (gt > p.tiles) gt = p.tiles;
    p.Gt = gt;
    p.lds = lds;
    return p;
}

static bool launch_pgemm(Engine* e, hipStream_t s, const WsCall& c) {
    if (c.K % kPgKC) return false;
    WsArgs a{};
    a.X = c.X; a.ldx = c.K; a.in_map = c.in_map; a.M = c.M; a.row0 = 0; a.K = c.K;
    a.gamma = (const uint16_t*)c.gamma; a.eps = c.eps; a.ss = c.ss; a.nss = c.nss;
    int tiles = 0;
    for (int i = 0; i < 3; ++i) {
        a.W[i] = i < c.nseg ? (const uint16_t*)c.W[i] : nullptr;
        a.seg_tiles[i] = i < c.nseg ? c.seg_rows[i] / 16 : 0;
        if (c.mode != kEpiSwiglu) tiles += a.seg_tiles[i];
    }
    if (c.mode == kEpiSwiglu) tiles = c.seg_rows[0] / 16;
    a.nseg = c.nseg; a.mode = c.mode; a.tiles = tiles;
    a.Y = c.Y; a.ldy = c.ldy; a.out_map = c.out_map; a.ss_out = c.ss_out;
    const int subs0 = c.mode == kEpiSwiglu ? 2 : 1;
    a.S = pg_split(c.M, tiles * 16, c.K, subs0);
    {
        // partials and counters must fit the workspace; else no K split
        const size_t nblkm = (size_t)(c.M + kPgRows - 1) / kPgRows;
        if (a.S > 1 && (nblkm * tiles * a.S * subs0 * 1024 > e->ws.ws_part_n || nblkm * tiles > e->ws.ws_cnt_n))
            a.S = 1;
    }
    a.part = c.part;
    a.cnt = c.cnt;
    a.H = c.H; a.Hkv = c.Hkv; a.hd = c.hd; a.row_pos = c.row_pos; a.row_seq = c.row_seq;
    a.rcos = c.rcos; a.rsin = c.rsin; a.qout = c.qout; a.kc = c.kc; a.vc = c.vc;
    a.cap = c.cap; a.max_batch = c.max_batch; a.layer = c.layer;
    a.ubias = c.ubias; a.ub_ld = c.ub_ld;
    const int subs = c.mode == kEpiSwiglu ? 2 : 1;
    const int nt = 4 * kPgTW / subs;
    const int nblk_m = (c.M + kPgRows - 1) / kPgRows;
    const int nblk_n = (tiles + nt - 1) / nt;
    const int nbs = 8 * nblk_m * ((nblk_n + 7) / 8);
    dim3 grid(nbs * a.S);
    const double wbytes = (double)tiles * 16 * subs * c.K * 2.0;
    ProfEntry* pe = prof_slot(e, kProfGemv, wbytes + (double)c.M * c.K * 4.0 + (double)c.M * tiles * 16 * 4.0);
    if (subs == 2) {
        if (pe) hipExtLaunchKernelGGL((k_pgemm<2>), grid, dim3(256), kPgLds, s, pe->a, pe->b, 0, a, nblk_m, nbs);
        else k_pgemm<2><<<grid, 256, kPgLds, s>>>(a, nblk_m, nbs);
    } else {
        if (pe) hipExtLaunchKernelGGL((k_pgemm<1>), grid, dim3(256), kPgLds, s, pe->a, pe->b, 0, a, nblk_m, nbs);
        else k_pgemm<1><<<grid, 256, kPgLds, s>>>(a, nblk_m, nbs);
    }
    if (pe) prof_commit(e);
    return true;
}

void launch_wsgemv(Engine* e, hipStream_t s, const WsCall& c) {
    // more than one 16-row group: the GEMM (weights read once per 64 rows, not per 16); also a
    // full 16-row group against a vocabulary-sized weight (the batched drafter steps' LM head),
    // which the GEMM streams faster
    int nrows = 0;
    for (int i = 0; i < c.nseg; ++i) nrows += c.seg_rows[i];
    if ((c.M > 16 || (c.M == 16 && nrows >= 32768)) && launch_pgemm(e, s, c)) return;
    for (int r0 = 0; r0 < c.M; r0 += 16) {
        int M = c.M - r0 < 16 ? c.M - r0 : 16;
        WsArgs a{};
        a.X = c.X; a.ldx = c.K; a.in_map = c.in_map; a.M = M; a.row0 = r0; a.K = c.K;
        a.gamma = (const uint16_t*)c.gamma; a.eps = c.eps; a.ss = c.ss; a.nss = c.nss;
        int tiles = 0;
        for (int i = 0; i < 3; ++i) {
            a.W[i] = i < c.nseg ? (const uint16_t*)c.W[i] : nullptr;
            a.seg_tiles[i] = i < c.nseg ? c.seg_rows[i] / 16 : 0;
            if (c.mode != kEpiSwiglu) tiles += a.seg_tiles[i];
        }
        if (c.mode == kEpiSwiglu) tiles = c.seg_rows[0] / 16;
        a.nseg = c.nseg; a.mode = c.mode; a.tiles = tiles;
        a.Y = c.Y; a.ldy = c.ldy; a.out_map = c.out_map; a.ss_out = c.ss_out;
        WsPlan p = ws_plan(M, tiles * 16, c.K, c.mode);
        a.KR = p.KR; a.S = p.S; a.Gt = p.Gt;
        a.part = c.part;
        a.cnt = c.cnt;
        a.H = c.H; a.Hkv = c.Hkv; a.hd = c.hd; a.row_pos = c.row_pos; a.row_seq = c.row_seq;
        a.rcos = c.rcos; a.rsin = c.rsin; a.qout = c.qout; a.kc = c.kc; a.vc = c.vc;
        a.cap = c.cap; a.max_batch = c.max_batch; a.layer = c.layer;
        a.ubias = c.ubias; a.ub_ld = c.ub_ld;
        int subs = c.mode == kEpiSwiglu ? 2 : 1;
        bool launched = false;
        if (p.S) {
            dim3 grid(p.S * p.Gt);
            double wbytes = (double)tiles * 16 * subs * c.K * 2.0;
            ProfEntry* pe = prof_slot(e, kProfGemv, wbytes + (double)M * c.K * 4.0 + (double)M * tiles * 16 * 4.0);
#define SD2_WS_CASE(NWV, ST, SB)                                                                     \
    if (!launched && p.NW == NWV && p.steps == ST && subs == SB) {                                    \
        if (pe)                                                                                       \
            hipExtLaunchKernelGGL((k_wsgemv<NWV, ST, SB>), grid, dim3(NWV * 64), p.lds, s, pe->a, pe->b, 0, a); \
        else                                                                                          \
            k_wsgemv<NWV, ST, SB><<<grid, NWV * 64, p.lds, s>>>(a);                                   \
        launched = true;                                                                              \
    }
#define SD2_WS_STEPS8(NWV, SB)                                                    \
    SD2_WS_CASE(NWV, 1, SB) SD2_WS_CASE(NWV, 2, SB) SD2_WS_CASE(NWV, 3, SB) SD2_WS_CASE(NWV, 4, SB) \
    SD2_WS_CASE(NWV, 5, SB) SD2_WS_CASE(NWV, 6, SB) SD2_WS_CASE(NWV, 7, SB) SD2_WS_CASE(NWV, 8, SB)
            SD2_WS_STEPS8(4, 1) SD2_WS_STEPS8(8, 1) SD2_WS_STEPS8(4, 2) SD2_WS_STEPS8(8, 2)
            SD2_WS_CASE(16, 1, 1) SD2_WS_CASE(16, 2, 1) SD2_WS_CASE(16, 3, 1) SD2_WS_CASE(16, 4, 1)
            SD2_WS_CASE(16, 1, 2) SD2_WS_CASE(16, 2, 2) SD2_WS_CASE(16, 3, 2) SD2_WS_CASE(16, 4, 2)
#undef SD2_WS_STEPS8
#undef SD2_WS_CASE
            if (pe && launched) prof_commit(e);
        }
        if (!launched && e) e->bad_launch = true;
    }
}

}  // namespace sd2
