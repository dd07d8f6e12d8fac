// Device-side helpers shared by the SD^2 kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd2 {

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

template <typename T>
__device__ __forceinline__ float load_scalar(const T* p, size_t i);
template <>
__device__ __forceinline__ float load_scalar<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_scalar<uint16_t>(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// (score, index) argmax with ties to the lower index.
struct ArgBest {
    float s;
    int i;
};
__device__ __forceinline__ bool better(float s, int i, float bs, int bi) {
    return s > bs || (s == bs && i < bi);
}
__device__ __forceinline__ ArgBest wave_argbest(ArgBest a) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        float s = __shfl_xor(a.s, o, kWave);
        int i = __shfl_xor(a.i, o, kWave);
        if (better(s, i, a.s, a.i)) { a.s = s; a.i = i; }
    }
    return a;
}

// Combine two (max, sum of exp(x - max)) pairs.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; s = s2; return; }
    if (m2 > m) { s = s * expf(m - m2) + s2; m = m2; }
    else { s = s + s2 * expf(m2 - m); }
}
__device__ __forceinline__ void wave_lse(float& m, float& s) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        float m2 = __shfl_xor(m, o, kWave);
        float s2 = __shfl_xor(s, o, kWave);
        lse_merge(m, s, m2, s2);
    }
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of
//   (x0,x1,x2,x3) -> (hi(B*x2) ^ x1 ^ k0, lo(B*x2), hi(A*x0) ^ x3 ^ k1, lo(A*x0))
// with A = 0xD2511F53, B = 0xCD9E8D57, the key advancing by the Weyl constants
// (0x9E3779B9, 0xBB67AE85) between rounds.
// ---------------------------------------------------------------------------
struct U4 {
    uint32_t x, y, z, w;
};
__device__ __forceinline__ U4 philox10(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint32_t a_lo = 0xD2511F53u * c.x, a_hi = __umulhi(0xD2511F53u, c.x);
        uint32_t b_lo = 0xCD9E8D57u * c.z, b_hi = __umulhi(0xCD9E8D57u, c.z);
        c = U4{b_hi ^ c.y ^ k0, b_lo, a_hi ^ c.w ^ k1, a_lo};
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// Random-stream purposes of the sampler (counter word 3 = purpose << 24 | sequence).
enum : uint32_t { kDraft = 1, kAccept = 2, kFinal = 3 };

__device__ __forceinline__ uint32_t rng_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t purpose,
                                             uint32_t seq, int word) {
    U4 r = philox10(U4{c0, c1, c2, (purpose << 24) | seq}, (uint32_t)seed, (uint32_t)(seed >> 32));
    return word == 0 ? r.x : word == 1 ? r.y : word == 2 ? r.z : r.w;
}

// Uniform in [2^-24, 1 - 2^-24]: top 23 bits + 1/2, scaled by 2^-23 (exact in fp32).
__device__ __forceinline__ float u01(uint32_t w) { return ((float)(w >> 9) + 0.5f) * (1.0f / 8388608.0f); }
__device__ __forceinline__ float gumbel(uint32_t w) { return -logf(-logf(u01(w))); }

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// Last-arriving workgroup hand-off inside one kernel, without a device-scope fence (on this
// part a release fence writes back the whole L2, which costs more than a kernel launch):
//   - every workgroup stores its partial with device-scope (write-through) stores and waits
//     until they have completed, then counts itself in with a device-scope atomic;
//   - the workgroup that counts in last reads all partials with ordinary loads.  Those lines
//     are read by nobody else during the kernel, so no stale copy of them can sit in the
//     reader's caches; the caches are invalidated at every kernel start.
// The last workgroup also resets the counter for the next launch.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void store_through(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Returns true in the last workgroup (uniform across the block).
__device__ __forceinline__ bool arrive_last(int32_t* cnt, int expected, int* flag_smem) {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        int prev = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag_smem = prev == expected - 1;
        if (prev == expected - 1) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    return *flag_smem != 0;
}

}  // namespace sd2
