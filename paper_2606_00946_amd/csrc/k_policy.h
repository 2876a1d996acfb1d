// Device-side pieces of the routing policy shared by the band selection and
// the route kernel.
#pragma once

#include "k_common.h"

namespace ls {

struct PolicyArgs {
    int32_t heuristic, count_col0, count_col1, kv_col, k_filter, cold;
    double theta_imbal, overload_k, prefix_tau, tau_sat, tau_ben, delta;
    uint64_t explore_thr;               // explore when the draw is below floor(epsilon * 2^32)
    const float* lo;                    // device [d] bounds, or null
    const float* hi;
};

struct PolicyStats {
    double limit;                       // mean + overload_k * std of the request counts
    int32_t imbalanced, saturated, any_inst_ood, pad;
};

// The splitmix64 mixing function (Steele, Lea and Flood, 2014).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

// Rendezvous top-K of a prefix group over N instances (Section 4.1, Consistent
// hashing based filtering): instance i weighs output i + 1 of splitmix64 seeded
// with the group key; C receives the K heaviest, heaviest first (ties to the
// lower id).  The whole wave calls it; C is uniform across the wave.
__device__ __forceinline__ int hrw_topk_wave(uint64_t key, int32_t N, int K, int32_t* C, int lane) {
    const int n = K < N ? K : N;
    for (int t = 0; t < n; ++t) {
        uint64_t bw = 0;
        int32_t bi = INT_MAX;
        for (int32_t i = lane; i < N; i += 64) {
            bool taken = false;
            for (int q = 0; q < t; ++q) taken |= (C[q] == i);
            if (taken) continue;
            const uint64_t w = mix64(key + 0x9e3779b97f4a7c15ull * (uint64_t)(i + 1));
            if (bi == INT_MAX || w > bw) { bw = w; bi = i; }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const uint64_t ow = shfl_xor_u64(bw, off);
            const int32_t oi = __shfl_xor(bi, off);
            if (oi != INT_MAX && (bi == INT_MAX || ow > bw || (ow == bw && oi < bi))) { bw = ow; bi = oi; }
        }
        C[t] = bi;
    }
    return n;
}

}  // namespace ls
