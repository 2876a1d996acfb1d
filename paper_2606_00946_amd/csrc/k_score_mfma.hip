// K2 on the matrix cores: bf16 reward model for every pair, then an exact
// decision by canonical rescoring of every candidate that could be the argmin.
//
// The reward model is one MLP shared by all instances (Section 4.1); in bf16
// mode its weights and every layer input are bf16, sums fp32.  The bulk of the
// work is the [pairs x h1] x [h1 x h2] hidden layer, a dense contraction, so it
// runs as v_mfma_f32_32x32x16_bf16 with rows = units and columns = pairs:
//   layer 1  C = the instance's layer-1 partial (b1 and the instance columns,
//            computed once per instance as the canonical chain), A = the
//            weights of the 5 derived columns, B = the pair's bf16 derived
//            columns: one k-step instead of d/16
//   layer 2  A = W2 fragments (LDS), B = bf16(relu(layer-1 accumulators)), C = b2
//   head     v_mfma_f32_16x16x32_bf16, A = [w3; |w3|; 0...], B = bf16(relu(layer-2
//            accumulators)) regrouped by v_permlane16_swap from the 32x32
//            B layout (16 units of one pair per lane half) into the 16x16x32 one
//            (8 units per 16-lane row), one row tile (K = 32) per instruction
// An accumulator of a 32x32 tile holds, in lane l and register r, unit
// 8(r/4) + 4(l/32) + r%4 of pair l%32.  The next layer's B operand needs, in
// lane l, eight consecutive k of pair l%32 -- so each layer's inputs are taken
// in that register order (perm_unit below) and the weights are stored with the
// same permutation of their input index: activations never leave registers.
//
// MFMA sums in an order of its own, so a bf16 activation near a rounding
// boundary can round differently than in the canonical fma chain.  Every pair
// therefore also gets an error scale E = kBandRel * (sum_j |w3_j| h2_j + |b3|)
// (the |w3| row of the head tile).  Per request, every pair whose interval
// [t - E, t + E] reaches the smallest t + E is rescored with the canonical
// chain, and the argmin runs over those canonical scores only; the chosen
// instance and its score are then the canonical ones whenever |t - t_canonical|
// <= E holds for the pairs left out.  The tests check that bound on every
// sampled pair with a margin.
#include "k_common.h"

namespace ls {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Input unit addressed by k-step s, lane half h, slot j of a B operand built
// straight from the previous layer's accumulators (s = 2*m_tile + half).
__host__ __device__ __forceinline__ int perm_unit(int s, int h, int j) {
    return 32 * (s >> 1) + 16 * (s & 1) + 8 * (j >> 2) + 4 * h + (j & 3);
}

__device__ __forceinline__ uint16_t bf16_bits(float x) { return (uint16_t)(__float_as_uint(bf16_rne(x)) >> 16); }

// ---------------------------------------------------------------------------
// fragment tables, rebuilt from the fp32 masters whenever the model changes
// ---------------------------------------------------------------------------
__global__ void prepare_mfma_kernel(MfmaLayout L, const float* __restrict__ master, uint16_t* __restrict__ frag16,
                                    float* __restrict__ frag32) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int d = L.d, h1 = L.h1;
    const float* W1 = master + L.m_w1;
    const float* W2 = master + L.m_w2;
    const float* W3 = master + L.m_w3;
    const int64_t nfrag = (L.w1_frags + L.w2_frags) * 512;
    if (t < nfrag) {
        const int j = (int)(t & 7);
        const int lane = (int)((t >> 3) & 63);
        const int64_t f = t >> 9;                       // fragment index
        const int m = lane & 31, h = lane >> 5;
        float v = 0.0f;
        if (f < L.w1_frags) {                            // [mt] : W1[32mt+m][d_inst+j], half 0, j < 5
            if (h == 0 && j < 5) v = W1[(int64_t)(32 * f + m) * d + L.d_inst + j];
        } else {                                         // [mt2][s(h1/16)] : W2[32mt2+m][perm(s,h,j)]
            const int64_t g = f - L.w1_frags;
            const int ks = h1 / 16;
            const int mt2 = (int)(g / ks), s = (int)(g % ks);
            v = W2[(int64_t)(32 * mt2 + m) * h1 + perm_unit(s, h, j)];
        }
        frag16[t] = bf16_bits(v);
    } else if (t < L.n16) {                              // head [mt][g][row][j]: row 0 w3, row 1 |w3|
        // the 16x16x32 A operand of row tile mt: k-group g holds the units of
        // k-step 2mt + (g & 1), lane half g >> 1 of the 32x32 B layout
        const int64_t e = t - nfrag;
        const int j = (int)(e & 7), row = (int)((e >> 3) & 1), g = (int)((e >> 4) & 3);
        const int mt = (int)(e >> 6);
        const float w = W3[perm_unit(2 * mt + (g & 1), g >> 1, j)];
        frag16[t] = bf16_bits(row == 0 ? w : fabsf(w));
    } else if (t < L.n16 + L.n32) {                      // b2
        frag32[t - L.n16] = master[L.m_b2 + (t - L.n16)];
    }
}

hipError_t launch_prepare_mfma(const MfmaLayout& L, const float* master, uint16_t* frag16, float* frag32,
                               hipStream_t s) {
    const int64_t n = L.n16 + L.n32;
    hipLaunchKernelGGL(prepare_mfma_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, L, master, frag16,
                       frag32);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// the MFMA scoring kernel: persistent; a workgroup works through units of 32
// requests x 16 instances (one instance group at a time)
// ---------------------------------------------------------------------------
constexpr int kGroupInst = 16;     // instances per group (columns n%16 of a tile)
constexpr int kUnitReq = 32;       // requests per unit: 8 waves x 2 tiles x 2

struct MfmaArgs {
    const bf16x8_t* __restrict__ w1frag;
    const bf16x8_t* __restrict__ w2frag;
    const bf16x8_t* __restrict__ hfrag;
    const float* __restrict__ b2;
    const float* __restrict__ b3;
    const float* __restrict__ part_t;             // [h1][N]: b1 + the instance columns, canonical
    const float* __restrict__ mu;
    const float* __restrict__ isig;
    const int64_t* __restrict__ req_off;
    const int32_t* __restrict__ prompt_len;
    const int32_t* __restrict__ overlap;
    float* __restrict__ scores;
    float* __restrict__ errb;
    int32_t R, N;
    int d_inst, block_tokens;
    float band_rel;
    int64_t n_rblocks;                             // ceil(R / 32)
    int64_t n_units;                               // ceil(N / 16) * n_rblocks
};

// bf16(relu(.)) of accumulator registers 8q .. 8q+7 as one B operand.  Rounding
// first and clamping the bf16 bit patterns at 0 as signed 16-bit integers is the
// same as relu-then-round for every non-NaN input (negative values and -0 map
// to +0), and takes one packed integer max per two values.
typedef short s16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ bf16x8_t relu_pack(const f32x16_t& acc, int q) {
    uint32_t w[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        f32x2_t v;
        v[0] = acc[8 * q + 2 * jj];
        v[1] = acc[8 * q + 2 * jj + 1];
        const bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
        s16x2_t si;
        __builtin_memcpy(&si, &p, sizeof si);
        si = __builtin_elementwise_max(si, s16x2_t{0, 0});
        __builtin_memcpy(&w[jj], &si, sizeof si);
    }
    bf16x8_t out;
    __builtin_memcpy(&out, w, sizeof out);
    return out;
}

// 16 consecutive accumulator-shaped floats: registers 4g .. 4g+3 from p[8g .. 8g+3].
__device__ __forceinline__ f32x16_t load_acc_rows(const float* p) {
    f32x16_t v;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float4 q = *reinterpret_cast<const float4*>(p + 8 * g);
        v[4 * g] = q.x; v[4 * g + 1] = q.y; v[4 * g + 2] = q.z; v[4 * g + 3] = q.w;
    }
    return v;
}

// Tile = 2 requests x 16 instances (lane column n: request n/16, instance
// n%16).  A wave scores two tiles per unit, of the same 16 instances, so every
// LDS read of weights, partials, biases and head rows serves both.  All of
// them sit in LDS (at h = 256: 8 + 128 KB of fragments, 16.6 KB of partials,
// 3 KB of biases and head rows); the partials are reloaded when the
// workgroup's units move on to the next instance group.
template <int MT>
__global__ __launch_bounds__(512, 1) void score_pairs_mfma_kernel(MfmaArgs A) {
    constexpr int H = 32 * MT;                 // h1 = h2
    constexpr int KS2 = 2 * MT;                // layer-2 k-steps: h1 / 16
    constexpr int QS = H + 4;                  // padded LDS row of one instance's partials
    constexpr int PT = 2;                      // tiles per wave and unit
    __shared__ bf16x8_t lds_w1[MT * 64];
    __shared__ bf16x8_t lds_w2[MT * KS2 * 64];
    __shared__ bf16x8_t lds_hd[2 * KS2 * 4];   // [mt][g][row], then as many zero fragments
    __shared__ __attribute__((aligned(16))) float lds_b2[H];
    __shared__ __attribute__((aligned(16))) float lds_q[kGroupInst * QS];
    const int tid = threadIdx.x;
    lds_fill<4>(lds_w1, MT * 64, [&](int f) { return A.w1frag[f]; });
    lds_fill<8>(lds_w2, MT * KS2 * 64, [&](int f) { return A.w2frag[f]; });
    for (int f = tid; f < 2 * KS2 * 4; f += blockDim.x) lds_hd[f] = f < KS2 * 4 ? A.hfrag[f] : bf16x8_t{};
    for (int f = tid; f < H; f += blockDim.x) lds_b2[f] = A.b2[f];

    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5, n = lane & 31;
    const int ni = n & 15, nr = n >> 4;
    const float b3 = A.b3[0];
    // head A operand (16x16x32): lane l holds row l % 16, k-group l / 16; rows 0
    // (w3) and 1 (|w3|) come from the table, the other lanes read the zero
    // fragments at the same offsets
    const int hrow = lane & 15, hgrp = lane >> 4;
    const bf16x8_t* hdl = lds_hd + (hrow < 2 ? hgrp * 2 + hrow : KS2 * 4);
    const int64_t u_begin = (int64_t)blockIdx.x * A.n_units / gridDim.x;
    const int64_t u_end = (int64_t)(blockIdx.x + 1) * A.n_units / gridDim.x;
    int64_t g_loaded = -1;
    for (int64_t u = u_begin; u < u_end; ++u) {
        const int64_t g = u / A.n_rblocks;
        const int64_t rb = u - g * A.n_rblocks;
        if (g != g_loaded) {                   // workgroup-uniform
            __syncthreads();
            for (int e = tid; e < kGroupInst * H; e += blockDim.x) {
                const int k = e / kGroupInst, q = e - k * kGroupInst;
                const int64_t ii = g * kGroupInst + q;
                lds_q[q * QS + k] = ii < A.N ? A.part_t[(int64_t)k * A.N + ii] : 0.0f;
            }
            __syncthreads();
            g_loaded = g;
        }
        const int64_t i = g * kGroupInst + ni;
        // The B operand of layer 1 holds a pair's five derived columns in lanes
        // 0-31 (k-group 0).  Lane (n, half) computes the columns of the pair of
        // its column n in tile p = half, and one permlane32 swap moves tile 1's
        // down to lanes 0-31.
        static_assert(PT == 2, "one pair tile per lane half");
        int64_t r[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p) r[p] = rb * kUnitReq + wave * (2 * PT) + 2 * p + nr;
        bf16x8_t xb[PT];
        {
            const int64_t rh = h ? r[1] : r[0];
            const bool valid = rh < A.R && i < A.N;
            const int64_t rr = valid ? rh : 0, ii = valid ? i : 0;
            float x[5], xt[5];
            derived_columns(A.prompt_len[rr], A.req_off[rr + 1] - A.req_off[rr], valid ? A.overlap[rr * A.N + ii] : 0,
                            A.block_tokens, x);
            normalise_tail<true>(x, A.mu, A.isig, A.d_inst, xt);
            bf16x8_t v{};
#pragma unroll
            for (int c = 0; c < 5; ++c) v[c] = (__bf16)xt[c];
            if (!valid) v = bf16x8_t{};
            uint32_t w[4], u[4];
            __builtin_memcpy(w, &v, sizeof w);
#pragma unroll
            for (int k = 0; k < 3; ++k) {                 // words 0-2 hold the five columns
                const auto sw = __builtin_amdgcn_permlane32_swap(w[k], w[k], false, false);
                u[k] = sw[1];                             // lanes 0-31: lane + 32's word
            }
            u[3] = 0u;
            bf16x8_t t1;
            __builtin_memcpy(&t1, u, sizeof t1);
            xb[0] = h == 0 ? v : bf16x8_t{};
            xb[1] = h == 0 ? t1 : bf16x8_t{};
        }

        // layer 1, one row tile at a time: acc = partial + W1_tail x_tail, then bf16(relu(.))
        const float* qrow = lds_q + ni * QS + 4 * h;
        bf16x8_t hb[PT][KS2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const f32x16_t c0 = load_acc_rows(qrow + 32 * mt);
            const bf16x8_t a = lds_w1[mt * 64 + lane];
#pragma unroll
            for (int p = 0; p < PT; ++p) {
                const f32x16_t acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xb[p], c0, 0, 0, 0);
                hb[p][2 * mt] = relu_pack(acc, 0);
                hb[p][2 * mt + 1] = relu_pack(acc, 1);
            }
        }

        // layer 2, one row tile at a time, each fed straight into the head:
        // row 0 = t, row 1 = sum_j |w3_j| h2_j
        // two 16x16 head tiles per pair tile: pairs 0-15 (its first request) and
        // 16-31 (its second); row 0 = t, row 1 = sum_j |w3_j| h2_j, in lanes 0-15
        f32x4_t hd[PT][2];
#pragma unroll
        for (int p = 0; p < PT; ++p) {
            hd[p][0] = f32x4_t{lane < 16 ? b3 : 0.0f, 0.0f, 0.0f, 0.0f};
            hd[p][1] = hd[p][0];
        }
        // The head of row tile mt runs inside the k-loop of row tile mt + 1
        // (pair tile 0 over k-steps 1-3, pair tile 1 over 4-6), so its VALU
        // work issues while the next tile's MFMAs execute.
        f32x16_t prev[PT];
        bf16x8_t fh_prev{};
        uint32_t pw0[PT][4], pw1[PT][4];
#pragma unroll
        for (int mt = 0; mt <= MT; ++mt) {
            const bool last = mt == MT;
            f32x16_t bias{};
            bf16x8_t fh{};
            const bf16x8_t* __restrict__ w2g = lds_w2;
            if (!last) {
                bias = load_acc_rows(lds_b2 + 32 * mt + 4 * h);
                fh = hdl[mt * 8];
                // a per-row-tile base keeps every read within the 16-bit immediate
                // offset of ds_read; the empty asm hides its value from the
                // optimiser, which would otherwise hoist one address register per
                // far fragment out of the loop
                uint32_t base = (uint32_t)(mt * KS2 * 64);
                asm volatile("" : "+s"(base));
                w2g = lds_w2 + base + lane;
            }
            f32x16_t acc[PT];
            // software pipeline: the next k-step's fragment is read while this
            // k-step's MFMAs run (the barriers pin that order)
            bf16x8_t a_cur{}, a_nxt{};
            if (!last) a_cur = w2g[0];
#pragma unroll
            for (int s = 0; s < (last || KS2 < 7 ? 7 : KS2); ++s) {
                if (!last && s + 1 < KS2) a_nxt = w2g[(s + 1) * 64];
                __builtin_amdgcn_sched_barrier(0);
                if (!last && s < KS2) {
#pragma unroll
                    for (int p = 0; p < PT; ++p)
                        acc[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_cur, hb[p][s], s == 0 ? bias : acc[p], 0, 0, 0);
                }
                if (mt > 0) {
                    // 16-lane rows of x0: units of k-step 2(mt-1), half 0, of pairs
                    // 0-15 and of 16-31, then half 1 of each; x1 the same for the
                    // next k-step.  The swap puts pairs 0-15's four 8-unit groups
                    // into b0, 16-31's into b1.
                    const int p = s < 4 ? 0 : 1, ph = s - 3 * p;
                    if (s >= 1 && s <= 6) {
                        if (ph == 1) {
                            const bf16x8_t x0 = relu_pack(prev[p], 0), x1 = relu_pack(prev[p], 1);
                            __builtin_memcpy(pw0[p], &x0, sizeof pw0[p]);
                            __builtin_memcpy(pw1[p], &x1, sizeof pw1[p]);
                        } else if (ph == 2) {
#pragma unroll
                            for (int k = 0; k < 4; ++k) {
                                const auto sw = __builtin_amdgcn_permlane16_swap(pw0[p][k], pw1[p][k], false, false);
                                pw0[p][k] = sw[0];
                                pw1[p][k] = sw[1];
                            }
                        } else {
                            bf16x8_t b0, b1;
                            __builtin_memcpy(&b0, pw0[p], sizeof b0);
                            __builtin_memcpy(&b1, pw1[p], sizeof b1);
                            hd[p][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh_prev, b0, hd[p][0], 0, 0, 0);
                            hd[p][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh_prev, b1, hd[p][1], 0, 0, 0);
                        }
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
                a_cur = a_nxt;
            }
            if (!last) {
#pragma unroll
                for (int p = 0; p < PT; ++p) prev[p] = acc[p];
                fh_prev = fh;
            }
        }
        // lane c < 16 holds instance c of both requests of each pair tile
        if (lane < 16 && i < A.N) {
#pragma unroll
            for (int p = 0; p < PT; ++p) {
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int64_t rq = r[p] + e;
                    if (rq < A.R) {
                        const int64_t q = rq * A.N + i;
                        A.scores[q] = hd[p][e][0];
                        A.errb[q] = A.band_rel * (hd[p][e][1] + fabsf(b3));
                    }
                }
            }
        }
    }
}

bool mfma_supported(const ModelDims& m) {
    return m.bf16 && m.L == 2 && (m.d == 16 || m.d == 32 || m.d == 48 || m.d == 64) &&
           (m.h1 == 64 || m.h1 == 128 || m.h1 == 256) && m.h1 == m.h2;
}

hipError_t launch_score_pairs_mfma(const ModelDims& m, const uint16_t* frag16, const float* frag32,
                                   const float* compute, const float* part_t, const float* mu,
                                   const float* inv_sigma, int32_t R, int32_t N, const int64_t* req_off,
                                   const int32_t* prompt_len, const int32_t* overlap, float* scores, float* errb,
                                   int n_cu, hipStream_t s) {
    if (R <= 0 || N <= 0) return hipSuccess;
    const MfmaLayout Lay = make_mfma_layout(m);
    MfmaArgs a;
    a.w1frag = reinterpret_cast<const bf16x8_t*>(frag16);
    a.w2frag = reinterpret_cast<const bf16x8_t*>(frag16 + Lay.w1_frags * 512);
    a.hfrag = reinterpret_cast<const bf16x8_t*>(frag16 + (Lay.w1_frags + Lay.w2_frags) * 512);
    a.b2 = frag32;
    a.b3 = compute + m.c_b3;
    a.part_t = part_t;
    a.mu = mu;
    a.isig = inv_sigma;
    a.req_off = req_off;
    a.prompt_len = prompt_len;
    a.overlap = overlap;
    a.scores = scores;
    a.errb = errb;
    a.R = R;
    a.N = N;
    a.d_inst = m.d_inst;
    a.block_tokens = m.block_tokens;
    a.band_rel = kBandRel;
    a.n_rblocks = ((int64_t)R + kUnitReq - 1) / kUnitReq;
    a.n_units = (((int64_t)N + kGroupInst - 1) / kGroupInst) * a.n_rblocks;
    int64_t grid = a.n_units < n_cu ? a.n_units : n_cu;
    if (grid < 1) grid = 1;
    if (m.h1 == 256)
        hipLaunchKernelGGL(score_pairs_mfma_kernel<8>, dim3((uint32_t)grid), dim3(512), 0, s, a);
    else if (m.h1 == 128)
        hipLaunchKernelGGL(score_pairs_mfma_kernel<4>, dim3((uint32_t)grid), dim3(512), 0, s, a);
    else
        hipLaunchKernelGGL(score_pairs_mfma_kernel<2>, dim3((uint32_t)grid), dim3(512), 0, s, a);
    return hipGetLastError();
}

}  // namespace ls
