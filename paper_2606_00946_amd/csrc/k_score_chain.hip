// K2 (canonical): the two-layer reward model's chains on the matrix cores.
//
// The canonical score of a pair (Section 4.1, the batched forward of Alg. 4) is
// a fixed sequence of fmaf roundings: layer 1 resumed from the instance partial
// over the five request/pair columns, each layer-2 unit from its bias over the
// layer-1 activations in ascending order, the head from b3 over the layer-2
// activations in ascending order (the chains of canonical_score).  The fp32
// matrix-core instruction v_mfma_f32_32x32x1_2b_f32 takes one input k per
// instruction and rounds each of its multiply-adds once, exactly as fmaf does
// (denormals kept), so stepping k in the chain's order reproduces every chain
// bit for bit: these scores equal the vector-ALU scorer's.
//
// A wave scores 32 pairs.  Both blocks of an instruction hold the same 32
// pairs (columns) and together 64 consecutive units (rows): lane l gives the A
// operand of unit 64 p + l, and lanes l and l + 32 give the same pair's B
// operand.  Accumulator register i of lane l then holds unit
// 64 p + 32 (i / 16) + 8 (i % 16 / 4) + 4 (l / 32) + i % 4 of pass p, pair l % 32.
//   layer 1: the accumulators start at the instance partials; five steps with
//            A = W1's column for that derived input, B = the pair's input;
//            ReLU (and bf16 rounding) into a wave-private LDS tile [pair][k];
//   layer 2: all h2 / 64 passes at once, accumulators from b2; per k one
//            coalesced 256-byte read of W2T row k per pass (A, held eight k
//            ahead) and one LDS read of four k of the pair's activations (B);
//   head:    ReLU (and bf16 rounding), then lanes 0-31 run the pair's chain,
//            taking units 4-7 of every 8 from lanes 32-63 (a lane shuffle).
#include <type_traits>

#include "k_common.h"

namespace ls {

namespace {

typedef float f32x32_t __attribute__((ext_vector_type(32)));

constexpr int kChainPairs = 32;   // pairs per wave

// LDS row stride of the activation tile: h1 rounded to 4, plus 4 when that is a
// multiple of 8 (16-byte reads of 32 rows without bank conflicts).
__host__ __device__ constexpr int chain_ldh(int h1) { return ((h1 + 3) & ~3) + ((((h1 + 3) >> 2) & 1) ? 0 : 4); }

template <bool BF>
__device__ __forceinline__ float act(float z) {
    const float a = relu(z);
    return BF ? bf16_rne_num(a) : a;
}

}  // namespace

// LIST: score the pairs list[0 .. *count) (pair indices r * N + i), with
// persistent waves that take 32 list entries at a time; otherwise every pair,
// one group of 32 per workgroup.  Up to h1 = 128 the tile leaves LDS for two
// waves per SIMD, so the kernels hold their registers to that; at 256, one.
template <bool BF, int H1, int H2, bool LIST>
__device__ __forceinline__ void chain_body(const PairModel& M, const float* __restrict__ mu,
                                           const float* __restrict__ isig, const float* __restrict__ part_t,
                                           int32_t R, int32_t N, const int64_t* __restrict__ req_off,
                                           const int32_t* __restrict__ prompt_len,
                                           const int32_t* __restrict__ overlap, int block_tokens,
                                           const int64_t* __restrict__ list, const uint32_t* __restrict__ count,
                                           float* __restrict__ scores) {
    static_assert(H1 % 64 == 0 && H2 % 64 == 0 && H1 <= 256 && H2 <= 256, "64-unit passes");
    constexpr int P1 = H1 / 64, P2 = H2 / 64, LDH = chain_ldh(H1);
    extern __shared__ __align__(16) float hl[];          // [kChainPairs][LDH]
    const int lane = threadIdx.x, col = lane & 31, hi = lane >> 5;
    const int64_t cnt = LIST ? (int64_t)*count : (int64_t)R * N;
    for (int64_t e0 = (int64_t)blockIdx.x * kChainPairs; e0 < cnt; e0 += (int64_t)gridDim.x * kChainPairs) {
    // the model's bases, opaque to the optimiser: their loads stay inside the
    // loop instead of holding b2, w3, W1 columns, W2T rows and partial addresses
    // in registers across tasks
    // (an opaque zero offset: the pointers keep their global address space)
    int32_t z0 = 0;
    asm volatile("" : "+s"(z0));
    const float *w1b = M.w1 + z0, *w2b = M.w2t + z0, *b2b = M.b2 + z0, *w3b = M.w3 + z0, *ptb = part_t + z0;
    const int32_t Nb = N + z0;
    const int64_t e = e0 + col < cnt ? e0 + col : cnt - 1;       // lanes past the end score a valid pair
    const int64_t q = LIST ? list[e] : e;
    const int64_t r = q / N;
    const int32_t inst = (int32_t)(q - r * N);
    float x[5], xt[5];
    derived_columns(prompt_len[r], req_off[r + 1] - req_off[r], overlap[q], block_tokens, x);
    normalise_tail<BF>(x, mu, isig, M.d_inst, xt);

    // layer 1, one 64-unit pass at a time, into the activation tile
    float* __restrict__ row = hl + col * LDH;
#pragma unroll
    for (int p = 0; p < P1; ++p) {
        f32x32_t acc;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            const int u = 64 * p + 32 * (i >> 4) + 8 * ((i & 15) >> 2) + 4 * hi + (i & 3);
            acc[i] = ptb[(uint32_t)(u * Nb + inst)];           // h1 N < 2^31
        }
        const float* __restrict__ w1 = w1b + (int64_t)(64 * p + lane) * M.d + M.d_inst;
        float a[5];
#pragma unroll
        for (int c = 0; c < 5; ++c) a[c] = w1[c];
#pragma unroll
        for (int c = 0; c < 5; ++c) acc = __builtin_amdgcn_mfma_f32_32x32x1f32(a[c], xt[c], acc, 0, 0, 0);
#pragma unroll
        for (int g = 0; g < 8; ++g) {          // registers 4 g .. 4 g + 3: four consecutive units
            const int u = 64 * p + 32 * (g >> 2) + 8 * (g & 3) + 4 * hi;
            *reinterpret_cast<float4*>(row + u) =
                make_float4(act<BF>(acc[4 * g]), act<BF>(acc[4 * g + 1]), act<BF>(acc[4 * g + 2]),
                            act<BF>(acc[4 * g + 3]));
        }
    }

    // layer 2: every pass at once
    f32x32_t acc[P2];
#pragma unroll
    for (int p = 0; p < P2; ++p)
#pragma unroll
        for (int i = 0; i < 32; ++i) acc[p][i] = b2b[64 * p + 32 * (i >> 4) + 8 * ((i & 15) >> 2) + 4 * hi + (i & 3)];
    const float* __restrict__ w2 = w2b + lane;              // W2T[k][64 p + lane] = w2[k * H2 + 64 p]
    constexpr int G = 8;                                    // inputs per group
    auto load = [&](float (&w)[G][P2], int k0) {
#pragma unroll
        for (int e = 0; e < G; ++e)
#pragma unroll
            for (int p = 0; p < P2; ++p) w[e][p] = w2[(int64_t)(k0 + e) * H2 + 64 * p];
    };
    auto step = [&](const float (&w)[G][P2], int k0) {
        float4 b[G / 4];
#pragma unroll
        for (int g = 0; g < G / 4; ++g) b[g] = *reinterpret_cast<const float4*>(row + k0 + 4 * g);
#pragma unroll
        for (int e = 0; e < G; ++e) {
            const float4 v = b[e >> 2];
            const float bv = (e & 3) == 0 ? v.x : (e & 3) == 1 ? v.y : (e & 3) == 2 ? v.z : v.w;
#pragma unroll
            for (int p = 0; p < P2; ++p) acc[p] = __builtin_amdgcn_mfma_f32_32x32x1f32(w[e][p], bv, acc[p], 0, 0, 0);
        }
    };
    static_assert(H1 % (2 * G) == 0, "whole double groups");
    float wa[G][P2], wb[G][P2];
    load(wa, 0);
#pragma unroll 1
    for (int k0 = 0; k0 < H1; k0 += 2 * G) {
        load(wb, k0 + G);
        step(wa, k0);
        if (k0 + 2 * G < H1) load(wa, k0 + 2 * G);
        step(wb, k0 + G);
    }

    // head: units in ascending order; lanes 0-31 hold units 0-3 of every 8, and
    // take units 4-7 from lanes 32-63
    float t = M.b3[0];
#pragma unroll
    for (int p = 0; p < P2; ++p)
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            const int u = 64 * p + 32 * (g >> 2) + 8 * (g & 3);
            float lo[4], up[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float h = act<BF>(acc[p][4 * g + e]);
                lo[e] = h;
                up[e] = __shfl_xor(h, 32);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) t = __builtin_fmaf(w3b[u + e], lo[e], t);
#pragma unroll
            for (int e = 0; e < 4; ++e) t = __builtin_fmaf(w3b[u + 4 + e], up[e], t);
        }
    if (hi == 0 && e0 + col < cnt) scores[q] = t;
    }
}

// Every pair, one group of 32 per workgroup.
template <bool BF, int H1, int H2>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(H1 <= 128 ? 2 : 1))) void score_chain_mfma_kernel(
    PairModel M, const float* __restrict__ mu, const float* __restrict__ isig, const float* __restrict__ part_t,
    int32_t R, int32_t N, const int64_t* __restrict__ req_off, const int32_t* __restrict__ prompt_len,
    const int32_t* __restrict__ overlap, int block_tokens, float* __restrict__ scores) {
    chain_body<BF, H1, H2, false>(M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, block_tokens, nullptr,
                                  nullptr, scores);
}

// The candidate band's rescoring: the pairs list[0 .. *count), persistent waves.
template <bool BF, int H1, int H2>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(H1 <= 128 ? 2 : 1))) void rescore_chain_mfma_kernel(
    PairModel M, const float* __restrict__ mu, const float* __restrict__ isig, const float* __restrict__ part_t,
    int32_t R, int32_t N, const int64_t* __restrict__ req_off, const int32_t* __restrict__ prompt_len,
    const int32_t* __restrict__ overlap, int block_tokens, const int64_t* __restrict__ list,
    const uint32_t* __restrict__ count, float* __restrict__ scores) {
    chain_body<BF, H1, H2, true>(M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, block_tokens, list, count,
                                 scores);
}

namespace {

template <bool BF, int H1, int H2>
hipError_t launch_chain(const PairModel& M, const float* mu, const float* isig, const float* part_t, int32_t R,
                        int32_t N, const int64_t* req_off, const int32_t* prompt_len, const int32_t* overlap,
                        int block_tokens, const int64_t* list, const uint32_t* count, int n_cu, float* scores,
                        hipStream_t s) {
    const size_t lds = sizeof(float) * kChainPairs * chain_ldh(H1);
    if (list) {
        // persistent: as many single-wave workgroups as the LDS lets every CU hold
        const int per_cu = (int)((160u << 10) / lds) < 8 ? (int)((160u << 10) / lds) : 8;
        hipLaunchKernelGGL((rescore_chain_mfma_kernel<BF, H1, H2>), dim3((uint32_t)(n_cu * per_cu)), dim3(64), lds,
                           s, M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, block_tokens, list, count,
                           scores);
    } else {
        const int64_t grid = ((int64_t)R * N + kChainPairs - 1) / kChainPairs;
        hipLaunchKernelGGL((score_chain_mfma_kernel<BF, H1, H2>), dim3((uint32_t)grid), dim3(64), lds, s, M, mu,
                           isig, part_t, R, N, req_off, prompt_len, overlap, block_tokens, scores);
    }
    return hipGetLastError();
}

template <bool BF>
hipError_t dispatch_chain(const ModelDims& m, const PairModel& M, const float* mu, const float* isig,
                          const float* part_t, int32_t R, int32_t N, const int64_t* req_off, const int32_t* prompt_len,
                          const int32_t* overlap, const int64_t* list, const uint32_t* count, int n_cu, float* scores,
                          hipStream_t s) {
    const int bt = m.block_tokens;
    if (m.h1 == 64)
        return launch_chain<BF, 64, 64>(M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, bt, list, count, n_cu,
                                        scores, s);
    if (m.h1 == 128)
        return launch_chain<BF, 128, 128>(M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, bt, list, count,
                                          n_cu, scores, s);
    return launch_chain<BF, 256, 256>(M, mu, isig, part_t, R, N, req_off, prompt_len, overlap, bt, list, count, n_cu,
                                      scores, s);
}

}  // namespace

bool chain_mfma_supported(const ModelDims& m) {
    return m.L == 2 && m.d == m.d_inst + 5 && m.h1 == m.h2 && (m.h1 == 64 || m.h1 == 128 || m.h1 == 256);
}

hipError_t launch_score_chain_mfma(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                                   const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                                   const int32_t* prompt_len, const int32_t* overlap, const int64_t* list,
                                   const uint32_t* count, int n_cu, float* scores, hipStream_t s) {
    if ((int64_t)R * N <= 0) return hipSuccess;
    if (!chain_mfma_supported(m) || (list == nullptr) != (count == nullptr)) return hipErrorInvalidValue;
    PairModel M{compute + m.c_w1, compute + m.c_w2t, compute + m.c_b2, compute + m.c_w3, compute + m.c_b3,
                m.d, m.d_inst, m.h1, m.h2};
    if (m.bf16)
        return dispatch_chain<true>(m, M, mu, inv_sigma, part_t, R, N, req_off, prompt_len, overlap, list, count, n_cu,
                                    scores, s);
    return dispatch_chain<false>(m, M, mu, inv_sigma, part_t, R, N, req_off, prompt_len, overlap, list, count, n_cu,
                                 scores, s);
}

}  // namespace ls
