// Message-passing litmus test of the library's fence-free hand-off protocol on the GPU it runs on
// (test infrastructure: built and run by tests/test_gpu_handoff.py).
//
// The protocol (persistent round program, split-K and span merges): a producer workgroup writes
// its values with device-scope write-through stores, waits for them to complete (vmcnt(0)), and
// then raises a counter with a relaxed device-scope atomic; a consumer polls that counter with
// relaxed atomic loads and then reads the values with ordinary global loads.  No fence is used.
// It relies on every such buffer being written once per launch before anybody reads it, so that
// no cache holds a stale copy (caches are invalidated at launch start).
//
// Here one launch holds one workgroup per compute unit.  In each of `rounds` rounds
// every workgroup writes a 4 KB message (its own lines, written once per launch), raises its
// flag, then waits (bounded) for the flag of a workgroup on another XCD and checks every word of
// that workgroup's message.  It reports words that did not match and waits that timed out.
// With --preread the consumer also reads the message lines before they are written (a
// violation of the write-once condition, reported for information, not asserted).
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "device_common.h"

namespace {

constexpr int kWords = 1024;  // floats per message
constexpr int kThreads = 256;

typedef const __attribute__((address_space(1))) float* gfp;
typedef __attribute__((address_space(1))) int32_t* gip;

__device__ __forceinline__ float word(int r, int w, int i) {
    return (float)(((unsigned)r * 7919u + (unsigned)w * 104729u + (unsigned)i * 31u) % 1000003u);
}

__global__ __launch_bounds__(kThreads) void k_litmus(float* data, int32_t* flags, int32_t* result, int rounds,
                                                     long spin_limit, int preread) {
    const int G = gridDim.x, w = blockIdx.x, tid = threadIdx.x;
    const int src = (w + G / 2 + 1) % G;  // G is a multiple of 8: src sits on another XCD
    __shared__ int arrived;
    __shared__ int bad_s;
    float keep = 0.f;
    for (int r = 0; r < rounds; ++r) {
        float* mine = data + ((size_t)r * G + w) * kWords;
        const float* theirs = data + ((size_t)r * G + src) * kWords;
        if (preread)
            for (int i = tid; i < kWords; i += kThreads) keep += *(gfp)(theirs + i);
        for (int i = tid; i < kWords; i += kThreads) sd2::store_through(mine + i, word(r, w, i));
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores have completed
        __syncthreads();
        if (tid == 0) {
            __hip_atomic_store((gip)(flags + (size_t)r * G + w), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            long s = 0;
            while (__hip_atomic_load((gip)(flags + (size_t)r * G + src), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0 &&
                   ++s < spin_limit)
                __builtin_amdgcn_s_sleep(1);
            arrived = s < spin_limit;
            bad_s = 0;
        }
        __syncthreads();
        if (!arrived) {
            if (tid == 0) atomicAdd(result + 1, 1);
            continue;
        }
        int bad = 0;
        for (int i = tid; i < kWords; i += kThreads) bad += *(gfp)(theirs + i) != word(r, src, i);
        if (bad) atomicAdd(&bad_s, bad);
        __syncthreads();
        if (tid == 0 && bad_s) atomicAdd(result, bad_s);
    }
    if (keep == -1.f) atomicAdd(result + 2, 1);  // keeps the control's reads alive
}

#define CK(x)                                                                                       \
    do {                                                                                            \
        hipError_t e_ = (x);                                                                        \
        if (e_ != hipSuccess) {                                                                     \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);          \
            return 2;                                                                               \
        }                                                                                           \
    } while (0)

}  // namespace

int main(int argc, char** argv) {
    int launches = 20, rounds = 64, preread = 0;
    for (int i = 1; i < argc; ++i) {
        if (!strcmp(argv[i], "--preread")) preread = 1;
        else if (!strcmp(argv[i], "--launches") && i + 1 < argc) launches = atoi(argv[++i]);
    }
    int dev = 0, cus = 0, occ = 0;
    CK(hipGetDevice(&dev));
    CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    CK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)k_litmus, kThreads, 0));
    if (cus < 16 || cus % 8 || occ < 1) {
        printf("litmus: skipped (compute units %d, workgroups per unit %d)\n", cus, occ);
        return 0;
    }
    const int G = cus;
    float* data;
    int32_t *flags, *result;
    CK(hipMalloc(&data, sizeof(float) * (size_t)rounds * G * kWords));
    CK(hipMalloc(&flags, sizeof(int32_t) * (size_t)rounds * G));
    CK(hipMalloc(&result, sizeof(int32_t) * 4));
    long total_bad = 0, total_timeouts = 0;
    const long spin_limit = 1L << 20;
    for (int l = 0; l < launches; ++l) {
        CK(hipMemset(data, 0, sizeof(float) * (size_t)rounds * G * kWords));
        CK(hipMemset(flags, 0, sizeof(int32_t) * (size_t)rounds * G));
        CK(hipMemset(result, 0, sizeof(int32_t) * 4));
        // one workgroup per compute unit (a plain launch: a cooperative one is refused while
        // another process holds the device; every wait is bounded and a timeout is reported)
        k_litmus<<<G, kThreads>>>(data, flags, result, rounds, spin_limit, preread);
        CK(hipGetLastError());
        int32_t h[4];
        CK(hipMemcpy(h, result, sizeof(h), hipMemcpyDeviceToHost));
        total_bad += h[0];
        total_timeouts += h[1];
    }
    printf("litmus: %s, %d launches x %d rounds x %d workgroups, %d words per message: %ld words wrong, %ld waits timed out\n",
           preread ? "lines read before they are written (control)" : "write-once lines", launches, rounds, G, kWords,
           total_bad, total_timeouts);
    CK(hipFree(data));
    CK(hipFree(flags));
    CK(hipFree(result));
    return 0;
}
