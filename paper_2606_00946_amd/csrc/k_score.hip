// K2/K3: pair features, shared reward model, per-request argmin.
//
// The reward model (Section 4.1, Request-instance reward model / Model
// architecture) is one MLP shared by every instance; it scores the row
// [instance state | request | pair] of each candidate and the request goes to
// the best prediction (Alg. 4: normalise, one batched forward, argmax reward;
// with the model predicting TTFT, argmin).
//
// Arithmetic order.  Every dot product is an fma chain that starts from the
// bias and walks the inputs in ascending order, with no other contraction, so
// a score is a deterministic function of its pair and identical pairs score
// identically.  Because the instance columns come first in the row, the first
// part of every layer-1 chain depends on the instance only: it is computed once
// per (instance, unit) and resumed per pair with the five request/pair columns.
// This leaves the chain, and so every rounding, unchanged.
//
// bf16 models (LS_BF16): weights and each layer's input activations are bf16
// values, products are exact in fp32, sums and biases stay fp32.
#include "k_common.h"

namespace ls {

// ---------------------------------------------------------------------------
// compute copy of the model
// ---------------------------------------------------------------------------
struct CopyArgs {
    int d, h1, h2;
    int64_t m_w1, m_b1, m_w2, m_b2, m_w3, m_b3;
    int64_t c_w1, c_b1, c_w2t, c_b2, c_w3, c_b3, c_w1t, n_compute;
    bool bf16;
};

__global__ void refresh_compute_kernel(CopyArgs a, const float* __restrict__ master, float* __restrict__ comp) {
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= a.n_compute) return;
    float v;
    bool weight = true;
    if (t < a.c_b1) {                                   // W1 [h1 x d]
        v = master[a.m_w1 + (t - a.c_w1)];
    } else if (t < a.c_w2t) {                           // b1
        v = master[a.m_b1 + (t - a.c_b1)];
        weight = false;
    } else if (t < a.c_b2) {                            // W2T[k][j] = W2[j][k]
        int64_t e = t - a.c_w2t;
        int64_t k = e / a.h2, j = e - k * a.h2;
        v = master[a.m_w2 + j * a.h1 + k];
    } else if (t < a.c_w3) {                            // b2
        v = master[a.m_b2 + (t - a.c_b2)];
        weight = false;
    } else if (t < a.c_b3) {                            // W3 [h2]
        v = master[a.m_w3 + (t - a.c_w3)];
    } else if (t < a.c_w1t) {                           // b3
        v = master[a.m_b3];
        weight = false;
    } else {                                            // W1T[c][k] = W1[k][c]
        int64_t e = t - a.c_w1t;
        int64_t c = e / a.h1, k = e - c * a.h1;
        v = master[a.m_w1 + k * a.d + c];
    }
    comp[t] = (weight && a.bf16) ? bf16_rne(v) : v;
}

// Other depths: every layer as W_l^T [in x out] then b_l, in layer order.
struct CopyLayers {
    int L;
    int in[4], out[4];
    int64_t m_w[4], m_b[4], c_wt[4], c_bl[4];
    int64_t n_compute;
    bool bf16;
};

__global__ void refresh_layers_kernel(CopyLayers a, const float* __restrict__ master, float* __restrict__ comp) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= a.n_compute) return;
    int l = 0;
    while (l < a.L && t >= a.c_wt[l + 1]) ++l;          // the layer whose segment holds t
    float v;
    bool weight;
    if (t < a.c_bl[l]) {                                // W_l^T[k][j] = W_l[j][k]
        const int64_t e = t - a.c_wt[l];
        const int64_t k = e / a.out[l], j = e - k * a.out[l];
        v = master[a.m_w[l] + j * a.in[l] + k];
        weight = true;
    } else {
        v = master[a.m_b[l] + (t - a.c_bl[l])];
        weight = false;
    }
    comp[t] = (weight && a.bf16) ? bf16_rne(v) : v;
}

hipError_t launch_refresh_compute_copy(const ModelDims& m, const float* master, float* compute, hipStream_t s) {
    const int64_t grid = (m.n_compute + 255) / 256;
    if (m.L != 2) {
        CopyLayers a{};
        a.L = m.L;
        for (int l = 0; l <= m.L; ++l) {
            a.in[l] = m.in_of(l);
            a.out[l] = m.out_of(l);
            a.m_w[l] = m.m_w[l];
            a.m_b[l] = m.m_b[l];
            a.c_wt[l] = m.c_wt[l];
            a.c_bl[l] = m.c_bl[l];
        }
        a.n_compute = m.n_compute;
        a.bf16 = m.bf16;
        hipLaunchKernelGGL(refresh_layers_kernel, dim3((uint32_t)grid), dim3(256), 0, s, a, master, compute);
        return hipGetLastError();
    }
    CopyArgs a{m.d, m.h1, m.h2, m.m_w1, m.m_b1, m.m_w2, m.m_b2, m.m_w3, m.m_b3,
               m.c_w1, m.c_b1, m.c_w2t, m.c_b2, m.c_w3, m.c_b3, m.c_w1t, m.n_compute, m.bf16};
    hipLaunchKernelGGL(refresh_compute_kernel, dim3((uint32_t)grid), dim3(256), 0, s, a, master, compute);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// layer-1 instance partials: part_t[k][i] = chain from b1[k] over the
// instance columns in ascending order.  A workgroup takes kPartInsts
// instances: their normalised columns go to LDS once per chunk of kPartCols
// columns, and each thread runs one unit's chains for all of them (independent
// chains; the unit's weights read eight columns ahead).
// ---------------------------------------------------------------------------
constexpr int kPartInsts = 8;
constexpr int kPartCols = 256;

template <bool BF>
__global__ __launch_bounds__(256) void instance_partial_kernel(const float* __restrict__ w1,
                                                               const float* __restrict__ b1,
                                                               const float* __restrict__ mu,
                                                               const float* __restrict__ isig,
                                                               const float* __restrict__ inst_feat, int d, int d_inst,
                                                               int h1, int32_t N, float* __restrict__ part_t) {
    __shared__ float xs[kPartInsts][kPartCols];
    const int32_t i0 = (int32_t)blockIdx.x * kPartInsts;
    const int tid = threadIdx.x;
    for (int kb = 0; kb < h1; kb += 256) {                        // uniform
        const int k = kb + tid;
        const bool kval = k < h1;
        const float* __restrict__ w = w1 + (int64_t)(kval ? k : 0) * d;
        float acc[kPartInsts];
        const float bk = kval ? b1[k] : 0.0f;
#pragma unroll
        for (int ii = 0; ii < kPartInsts; ++ii) acc[ii] = bk;
        for (int c0 = 0; c0 < d_inst; c0 += kPartCols) {          // uniform
            const int nc = min(kPartCols, d_inst - c0);
            __syncthreads();                                      // the last chunk's reads are done
            for (int e = tid; e < kPartInsts * kPartCols; e += 256) {
                const int ii = e / kPartCols, c = e - ii * kPartCols;
                const int32_t i = i0 + ii;
                float x = 0.0f;
                if (i < N && c < nc) {
                    x = __fmul_rn(__fsub_rn(inst_feat[(int64_t)i * d_inst + c0 + c], mu[c0 + c]), isig[c0 + c]);
                    if (BF) x = bf16_rne(x);
                }
                xs[ii][c] = x;
            }
            __syncthreads();
            int c = 0;
            for (; c + 8 <= nc; c += 8) {
                float wc[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) wc[j] = w[c0 + c + j];
#pragma unroll
                for (int j = 0; j < 8; ++j)
#pragma unroll
                    for (int ii = 0; ii < kPartInsts; ++ii) acc[ii] = __builtin_fmaf(wc[j], xs[ii][c + j], acc[ii]);
            }
            for (; c < nc; ++c) {
                const float wc = w[c0 + c];
#pragma unroll
                for (int ii = 0; ii < kPartInsts; ++ii) acc[ii] = __builtin_fmaf(wc, xs[ii][c], acc[ii]);
            }
        }
        if (kval) {
#pragma unroll
            for (int ii = 0; ii < kPartInsts; ++ii)
                if (i0 + ii < N) part_t[(int64_t)k * N + i0 + ii] = acc[ii];
        }
    }
}

hipError_t launch_instance_partial(const ModelDims& m, const float* compute, const float* mu,
                                   const float* inv_sigma, const float* inst_feat, int32_t N, float* part_t,
                                   hipStream_t s) {
    const int64_t grid = ((int64_t)N + kPartInsts - 1) / kPartInsts;
    if (grid == 0) return hipSuccess;
    if (m.bf16)
        hipLaunchKernelGGL(instance_partial_kernel<true>, dim3((uint32_t)grid), dim3(256), 0, s, compute + m.c_w1,
                           compute + m.c_b1, mu, inv_sigma, inst_feat, m.d, m.d_inst, m.h1, N, part_t);
    else
        hipLaunchKernelGGL(instance_partial_kernel<false>, dim3((uint32_t)grid), dim3(256), 0, s, compute + m.c_w1,
                           compute + m.c_b1, mu, inv_sigma, inst_feat, m.d, m.d_inst, m.h1, N, part_t);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pair scoring: one lane per pair, weights uniform across the wave
// ---------------------------------------------------------------------------
template <bool BF>
__global__ __launch_bounds__(256) void score_pairs_kernel(PairModel M, const float* __restrict__ mu,
                                                          const float* __restrict__ isig,
                                                          const float* __restrict__ part_t, int32_t R, int32_t N,
                                                          const int64_t* __restrict__ req_off,
                                                          const int32_t* __restrict__ prompt_len,
                                                          const int32_t* __restrict__ overlap, int block_tokens,
                                                          float* __restrict__ scores) {
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)R * N;
    const bool valid = p < total;
    const int64_t pp = valid ? p : 0;
    const int64_t r = pp / N, i = pp - r * N;
    float x[5], xt[5];
    derived_columns(prompt_len[r], req_off[r + 1] - req_off[r], overlap[pp], block_tokens, x);
    normalise_tail<BF>(x, mu, isig, M.d_inst, xt);
    const float t = canonical_score<BF>(M, part_t + i, N, xt);
    if (valid) scores[p] = t;
}

hipError_t launch_score_pairs(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                              const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                              const int32_t* prompt_len, const int32_t* overlap, float* scores, hipStream_t s) {
    int64_t total = (int64_t)R * N;
    if (total <= 0) return hipSuccess;
    PairModel M{compute + m.c_w1, compute + m.c_w2t, compute + m.c_b2, compute + m.c_w3, compute + m.c_b3,
                m.d, m.d_inst, m.h1, m.h2};
    int64_t grid = (total + 255) / 256;
    if (m.bf16)
        hipLaunchKernelGGL(score_pairs_kernel<true>, dim3((uint32_t)grid), dim3(256), 0, s, M, mu, inv_sigma, part_t,
                           R, N, req_off, prompt_len, overlap, m.block_tokens, scores);
    else
        hipLaunchKernelGGL(score_pairs_kernel<false>, dim3((uint32_t)grid), dim3(256), 0, s, M, mu, inv_sigma, part_t,
                           R, N, req_off, prompt_len, overlap, m.block_tokens, scores);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// K3: per-request argmin, one wave per request
// ---------------------------------------------------------------------------
// With a band (VEC: N a multiple of 4, the flags word-aligned) lane l reads the
// flags of pairs 4l .. 4l + 3 of each chunk of 256 as one word.
template <bool VEC>
__global__ __launch_bounds__(256) void argmin_kernel(int32_t R, int32_t N, int d, int d_inst, int block_tokens,
                                                     const float* __restrict__ scores,
                                                     const uint8_t* __restrict__ band,
                                                     const int64_t* __restrict__ req_off,
                                                     const int32_t* __restrict__ prompt_len,
                                                     const int32_t* __restrict__ overlap,
                                                     const float* __restrict__ inst_feat,
                                                     int32_t* __restrict__ chosen, float* __restrict__ min_ttft,
                                                     float* __restrict__ feat_out) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (r >= R) return;
    const float* __restrict__ s = scores + r * N;
    float bs = 0.0f;
    int bi = INT_MAX;
    if constexpr (VEC) {
        for (int i = 4 * lane; i < N; i += 256) {
            const uint32_t bits = *reinterpret_cast<const uint32_t*>(band + r * N + i);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (!((bits >> (8 * j)) & 0xFFu)) continue;      // only candidates that were rescored
                const float v = s[i + j];
                if (better(v, i + j, bs, bi)) { bs = v; bi = i + j; }
            }
        }
    } else {
        for (int i = lane; i < N; i += 64) {
            if (band && !band[r * N + i]) continue;          // only candidates that were rescored
            float v = s[i];
            if (better(v, i, bs, bi)) { bs = v; bi = i; }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        float os = __shfl_xor(bs, off);
        int oi = __shfl_xor(bi, off);
        if (better(os, oi, bs, bi)) { bs = os; bi = oi; }
    }
    if (lane == 0) {
        chosen[r] = bi;
        if (min_ttft) min_ttft[r] = bs;
    }
    if (feat_out) {
        float x[5];
        derived_columns(prompt_len[r], req_off[r + 1] - req_off[r], overlap[r * N + bi], block_tokens, x);
        for (int c = lane; c < d; c += 64) {
            const float v = c < d_inst ? inst_feat[(int64_t)bi * d_inst + c] : x[c - d_inst];
            feat_out[r * d + c] = v;
        }
    }
}

hipError_t launch_argmin(const ModelDims& m, int32_t R, int32_t N, const float* scores, const uint8_t* band,
                         const int64_t* req_off, const int32_t* prompt_len, const int32_t* overlap,
                         const float* inst_feat, int32_t* chosen, float* min_ttft, float* feat_out, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    int64_t grid = ((int64_t)R + 3) / 4;
    if (band && N % 4 == 0 && (uintptr_t)band % 4 == 0)
        hipLaunchKernelGGL(argmin_kernel<true>, dim3((uint32_t)grid), dim3(256), 0, s, R, N, m.d, m.d_inst,
                           m.block_tokens, scores, band, req_off, prompt_len, overlap, inst_feat, chosen, min_ttft,
                           feat_out);
    else
        hipLaunchKernelGGL(argmin_kernel<false>, dim3((uint32_t)grid), dim3(256), 0, s, R, N, m.d, m.d_inst,
                           m.block_tokens, scores, band, req_off, prompt_len, overlap, inst_feat, chosen, min_ttft,
                           feat_out);
    return hipGetLastError();
}

}  // namespace ls
