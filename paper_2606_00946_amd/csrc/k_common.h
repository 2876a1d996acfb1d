// Device helpers shared by the scoring kernels: bf16 rounding, ReLU, the
// lexicographic (score, id) order of the argmin, and the canonical per-pair
// evaluation of the reward model (fma chains from the bias in ascending input
// order, layer 1 resumed from the per-instance partial).
#pragma once

#include <climits>

#include "ls_internal.h"

namespace ls {

// Round to the nearest bf16 value, ties to even (bits of a binary32).
__device__ __forceinline__ float bf16_rne(float x) {
    if (x != x) return x;
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

// Same, for values known not to be NaN (ReLU outputs).
__device__ __forceinline__ float bf16_rne_num(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

__device__ __forceinline__ float relu(float z) { return z > 0.0f ? z : 0.0f; }

// Workgroup-cooperative fill of a shared-memory array: dst[e] = get(e) for e in
// [0, n).  Each thread issues INFLIGHT loads before storing any of them, so the
// fill costs one memory round trip per INFLIGHT elements per thread rather than
// one per element (a plain strided loop waits for every load before its store).
template <int INFLIGHT, class T, class Get>
__device__ __forceinline__ void lds_fill(T* dst, int n, Get get) {
    const int T_ = (int)blockDim.x;
    for (int e0 = (int)threadIdx.x; e0 < n; e0 += T_ * INFLIGHT) {
        T v[INFLIGHT];
#pragma unroll
        for (int j = 0; j < INFLIGHT; ++j)
            if (e0 + j * T_ < n) v[j] = get(e0 + j * T_);
#pragma unroll
        for (int j = 0; j < INFLIGHT; ++j)
            if (e0 + j * T_ < n) dst[e0 + j * T_] = v[j];
    }
}

struct PairModel {
    const float* __restrict__ w1;    // [h1 x d]
    const float* __restrict__ w2t;   // [h1 x h2]
    const float* __restrict__ b2;    // [h2]
    const float* __restrict__ w3;    // [h2]
    const float* __restrict__ b3;    // [1]
    int d, d_inst, h1, h2;
};

// U consecutive layer-2 units starting at jb, then their head terms in order.
template <bool BF, int U>
__device__ __forceinline__ float unit_block(const PairModel& M, const float* __restrict__ part_i, int32_t N,
                                            const float xt[5], int jb, float t) {
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = M.b2[jb + u];
#pragma unroll 4
    for (int k = 0; k < M.h1; ++k) {
        float z = part_i[(int64_t)k * N];
        const float* __restrict__ w1 = M.w1 + (int64_t)k * M.d + M.d_inst;
#pragma unroll
        for (int c = 0; c < 5; ++c) z = __builtin_fmaf(w1[c], xt[c], z);
        float a = relu(z);
        if (BF) a = bf16_rne_num(a);
        const float* __restrict__ w2 = M.w2t + (int64_t)k * M.h2 + jb;
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] = __builtin_fmaf(w2[u], a, acc[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float hh = relu(acc[u]);
        if (BF) hh = bf16_rne_num(hh);
        t = __builtin_fmaf(M.w3[jb + u], hh, t);
    }
    return t;
}

// The five derived columns of a pair row: prompt tokens L, hashed blocks n,
// overlap l, hit ratio kappa = bt*l/L (0 when L = 0), uncached tokens L - bt*l.
__device__ __forceinline__ void derived_columns(int32_t L, int64_t n, int32_t l, int block_tokens, float x[5]) {
    const int64_t hit = (int64_t)block_tokens * l;
    x[0] = (float)L;
    x[1] = (float)n;
    x[2] = (float)l;
    // divide unconditionally by a safe denominator, then select: no branch
    const float ratio = (float)hit / (float)(L == 0 ? 1 : L);
    x[3] = (L == 0) ? 0.0f : ratio;
    x[4] = (float)((int64_t)L - hit);
}

// z-score of the derived columns: (x - mu) * inv_sigma, two roundings, then bf16 in bf16 mode.
template <bool BF>
__device__ __forceinline__ void normalise_tail(const float x[5], const float* __restrict__ mu,
                                               const float* __restrict__ isig, int d_inst, float xt[5]) {
#pragma unroll
    for (int c = 0; c < 5; ++c) {
        float v = __fmul_rn(__fsub_rn(x[c], mu[d_inst + c]), isig[d_inst + c]);
        xt[c] = BF ? bf16_rne(v) : v;
    }
}

// Canonical score of one pair: layer 1 resumed from the instance partial, the
// layer-2 chains in blocks of units, and the head chain in ascending unit order.
template <bool BF>
__device__ __forceinline__ float canonical_score(const PairModel& M, const float* __restrict__ part_i, int32_t N,
                                                 const float xt[5]) {
    float t = M.b3[0];
    int jb = 0;
    for (; jb + 32 <= M.h2; jb += 32) t = unit_block<BF, 32>(M, part_i, N, xt, jb, t);
    if (jb + 16 <= M.h2) { t = unit_block<BF, 16>(M, part_i, N, xt, jb, t); jb += 16; }
    if (jb + 8 <= M.h2) { t = unit_block<BF, 8>(M, part_i, N, xt, jb, t); jb += 8; }
    if (jb + 4 <= M.h2) { t = unit_block<BF, 4>(M, part_i, N, xt, jb, t); jb += 4; }
    if (jb + 2 <= M.h2) { t = unit_block<BF, 2>(M, part_i, N, xt, jb, t); jb += 2; }
    if (jb + 1 <= M.h2) { t = unit_block<BF, 1>(M, part_i, N, xt, jb, t); jb += 1; }
    return t;
}

// Lexicographic order on (score, id): -0 equals +0, NaN after +inf, ties to the
// lower id; id INT_MAX marks "no candidate yet".
__device__ __forceinline__ bool better(float a, int ia, float b, int ib) {
    if (ia == INT_MAX) return false;
    if (ib == INT_MAX) return true;
    const bool an = a != a, bn = b != b;
    if (an) return bn && ia < ib;
    if (bn) return true;
    if (a < b) return true;
    if (a > b) return false;
    return ia < ib;
}

}  // namespace ls
