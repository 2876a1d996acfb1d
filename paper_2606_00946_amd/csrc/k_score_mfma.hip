// K2 on the matrix cores: bf16 reward model for every pair, then an exact
// decision by canonical rescoring of every candidate that could be the argmin.
//
// The reward model is one MLP shared by all instances (Section 4.1); in bf16
// mode its weights and every layer input are bf16, sums fp32.  The bulk of the
// work is the [pairs x h1] x [h1 x h2] hidden layer, a dense contraction, so it
// runs as v_mfma_f32_32x32x16_bf16 with rows = units and columns = pairs:
//   layer 1  A = W1 fragments, B = normalised bf16 pair rows, C = b1
//   layer 2  A = W2 fragments (LDS), B = bf16(relu(layer-1 accumulators))
//   head     A = [w3; |w3|; 0...], B = bf16(relu(layer-2 accumulators))
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
        if (f < L.w1_frags) {                            // [s(4)][mt] : W1[32mt+m][16s+8h+j]
            const int mt1 = h1 / 32;
            const int s = (int)(f / mt1), mt = (int)(f % mt1);
            const int c = 16 * s + 8 * h + j;
            if (c < d) v = W1[(int64_t)(32 * mt + m) * d + c];
        } else {                                         // [mt2][s(h1/16)] : W2[32mt2+m][perm(s,h,j)]
            const int64_t g = f - L.w1_frags;
            const int ks = h1 / 16;
            const int mt2 = (int)(g / ks), s = (int)(g % ks);
            v = W2[(int64_t)(32 * mt2 + m) * h1 + perm_unit(s, h, j)];
        }
        frag16[t] = bf16_bits(v);
    } else if (t < L.n16) {                              // head fragments [s(h2/16)][lane][j]: rows w3, |w3|
        const int64_t e = t - nfrag;
        const int j = (int)(e & 7), lane = (int)((e >> 3) & 63);
        const int s = (int)(e >> 9);
        const int m = lane & 31, h = lane >> 5;
        const float w = W3[perm_unit(s, h, j)];
        frag16[t] = bf16_bits(m == 0 ? w : m == 1 ? fabsf(w) : 0.0f);
    } else if (t < L.n16 + L.n32) {                      // bias fragments [mt][h][r] for b1 then b2
        const int64_t e = t - L.n16;
        const int r = (int)(e & 15), h = (int)((e >> 4) & 1);
        const int64_t mt = e >> 5;
        const int unit_in_tile = 8 * (r >> 2) + 4 * h + (r & 3);
        const int mt1 = h1 / 32;
        float v;
        if (mt < mt1) v = master[L.m_b1 + 32 * mt + unit_in_tile];
        else v = master[L.m_b2 + 32 * (mt - mt1) + unit_in_tile];
        frag32[e] = v;
    }
}

hipError_t launch_prepare_mfma(const MfmaLayout& L, const float* master, uint16_t* frag16, float* frag32,
                               hipStream_t s) {
    const int64_t n = L.n16 + L.n32;
    hipLaunchKernelGGL(prepare_mfma_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, L, master, frag16,
                       frag32);
    return hipGetLastError();
}

// Normalised bf16 instance columns, 64 per instance (zero past d_inst).
__global__ void instance_rows_kernel(const float* __restrict__ inst_feat, const float* __restrict__ mu,
                                     const float* __restrict__ isig, int d_inst, int32_t N,
                                     uint16_t* __restrict__ xinst) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)N * 64) return;
    const int64_t i = t >> 6;
    const int c = (int)(t & 63);
    float v = 0.0f;
    if (c < d_inst) v = __fmul_rn(__fsub_rn(inst_feat[i * d_inst + c], mu[c]), isig[c]);
    xinst[t] = bf16_bits(v);
}

hipError_t launch_instance_rows(const ModelDims& m, const float* mu, const float* inv_sigma, const float* inst_feat,
                                int32_t N, uint16_t* xinst, hipStream_t s) {
    const int64_t n = (int64_t)N * 64;
    hipLaunchKernelGGL(instance_rows_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, inst_feat, mu,
                       inv_sigma, m.d_inst, N, xinst);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// the MFMA scoring kernel: persistent, one 32-pair tile per wave at a time
// ---------------------------------------------------------------------------
struct MfmaArgs {
    const bf16x8_t* __restrict__ w1frag;
    const bf16x8_t* __restrict__ w2frag;
    const bf16x8_t* __restrict__ hfrag;
    const float* __restrict__ b1frag;
    const float* __restrict__ b2frag;
    const float* __restrict__ b3;
    const uint16_t* __restrict__ xinst;
    const float* __restrict__ mu;
    const float* __restrict__ isig;
    const int64_t* __restrict__ req_off;
    const int32_t* __restrict__ prompt_len;
    const int32_t* __restrict__ overlap;
    float* __restrict__ scores;
    float* __restrict__ errb;
    int32_t R, N;
    int d, d_inst, block_tokens;
    float band_rel;
};

__device__ __forceinline__ f32x16_t load_bias(const float* __restrict__ p) {
    const float4* q = reinterpret_cast<const float4*>(p);
    float4 a = q[0], b = q[1], c = q[2], e = q[3];
    f32x16_t v;
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    v[8] = c.x; v[9] = c.y; v[10] = c.z; v[11] = c.w;
    v[12] = e.x; v[13] = e.y; v[14] = e.z; v[15] = e.w;
    return v;
}

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

// One wave scores two tiles of 32 pairs (32 consecutive instances of one
// request each; consecutive tiles in request-major order) per pass; the eight
// waves of a workgroup share the W1 and W2 fragments in LDS (32 + 128 KB at
// h = 256).  Every weight fragment read from LDS feeds one MFMA per tile, and
// every bias and head fragment read serves both tiles.  Each layer runs one
// row tile at a time, so that few accumulators are live beside the second
// layer's 2 x h1 bf16 inputs.
template <int MT1, int MT2, int D>
__global__ __launch_bounds__(512, 1) void score_pairs_mfma_kernel(MfmaArgs A) {
    static_assert(MT1 == MT2, "square hidden layers");
    constexpr int KS2 = 2 * MT1;               // layer-2 k-steps: h1 / 16
    constexpr int D_INST = D - 5;
    constexpr int NW1 = 4 * MT1 * 64, NW2 = MT2 * KS2 * 64;
    constexpr int PT = 2;                      // tiles per pass
    __shared__ bf16x8_t lds_w1[NW1];
    __shared__ bf16x8_t lds_w2[NW2];
    for (int f = threadIdx.x; f < NW1; f += blockDim.x) lds_w1[f] = A.w1frag[f];
    for (int f = threadIdx.x; f < NW2; f += blockDim.x) lds_w2[f] = A.w2frag[f];
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int waves = blockDim.x >> 6;
    const int h = lane >> 5, n = lane & 31;
    const int tiles_per_req = (A.N + 31) >> 5;
    const int64_t n_tiles = (int64_t)A.R * tiles_per_req;
    const int64_t n_passes = (n_tiles + PT - 1) / PT;
    const float b3 = A.b3[0];
    const bf16x8_t* __restrict__ hf = A.hfrag + lane;
    const bf16x8_t* __restrict__ w1l = lds_w1 + lane;
    for (int64_t pass = (int64_t)blockIdx.x * waves + (threadIdx.x >> 6); pass < n_passes;
         pass += (int64_t)gridDim.x * waves) {
        int64_t r[PT];
        int i[PT];
        bool valid[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p) {                 // a second tile past the end computes on tile 0's data
            const int64_t t = PT * pass + p;
            const int64_t tt = t < n_tiles ? t : 0;
            r[p] = tt / tiles_per_req;
            i[p] = (int)(tt - r[p] * tiles_per_req) * 32 + n;
            valid[p] = t < n_tiles && i[p] < A.N;
        }

        // layer-1 B operands: the pairs' normalised bf16 rows
        bf16x8_t xb[PT][4];
#pragma unroll
        for (int p = 0; p < PT; ++p) {
            const int ii = valid[p] ? i[p] : 0;
            float x[5], xt[5];
            derived_columns(A.prompt_len[r[p]], A.req_off[r[p] + 1] - A.req_off[r[p]],
                            valid[p] ? A.overlap[r[p] * A.N + ii] : 0, A.block_tokens, x);
            normalise_tail<true>(x, A.mu, A.isig, D_INST, xt);
            const bf16x8_t* row = reinterpret_cast<const bf16x8_t*>(A.xinst + (int64_t)ii * 64);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                bf16x8_t v = row[2 * s + h];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int c0 = 16 * s + j - D_INST;       // derived column held by half 0
                    const int c1 = c0 + 8;                    // ... by half 1
                    if (c0 >= 0 && c0 < 5 && h == 0) v[j] = (__bf16)xt[c0 < 5 ? c0 : 0];
                    if (c1 >= 0 && c1 < 5 && h == 1) v[j] = (__bf16)xt[c1 < 5 ? c1 : 0];
                }
                xb[p][s] = valid[p] ? v : bf16x8_t{};
            }
        }

        // layer 1, one row tile at a time: acc = b1 + W1 x, then bf16(relu(.))
        bf16x8_t hb[PT][KS2];
#pragma unroll
        for (int mt = 0; mt < MT1; ++mt) {
            const f32x16_t bias = load_bias(A.b1frag + (mt * 2 + h) * 16);
            f32x16_t acc[PT];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const bf16x8_t a = w1l[(s * MT1 + mt) * 64];
#pragma unroll
                for (int p = 0; p < PT; ++p)
                    acc[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xb[p][s], s == 0 ? bias : acc[p], 0, 0, 0);
            }
#pragma unroll
            for (int p = 0; p < PT; ++p) {
                hb[p][2 * mt] = relu_pack(acc[p], 0);
                hb[p][2 * mt + 1] = relu_pack(acc[p], 1);
            }
        }

        // layer 2, one row tile at a time, each fed straight into the head:
        // row 0 = t, row 1 = sum_j |w3_j| h2_j
        f32x16_t hd[PT];
#pragma unroll
        for (int p = 0; p < PT; ++p) {
            hd[p] = f32x16_t{};
            hd[p][0] = h == 0 ? b3 : 0.0f;
        }
#pragma unroll
        for (int mt = 0; mt < MT2; ++mt) {
            const f32x16_t bias = load_bias(A.b2frag + (mt * 2 + h) * 16);
            // a per-row-tile base keeps every read within the 16-bit immediate
            // offset of ds_read; the empty asm hides its value from the
            // optimiser, which would otherwise hoist one address register per
            // far fragment out of the loop
            uint32_t base = (uint32_t)(mt * KS2 * 64);
            asm volatile("" : "+s"(base));
            const bf16x8_t* __restrict__ w2g = lds_w2 + base + lane;
            f32x16_t acc[PT];
            // software pipeline: the next k-step's fragment is read while this
            // k-step's MFMAs run (the barriers pin that order)
            bf16x8_t a_cur = w2g[0], a_nxt;
#pragma unroll
            for (int s = 0; s < KS2; ++s) {
                if (s + 1 < KS2) a_nxt = w2g[(s + 1) * 64];
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int p = 0; p < PT; ++p)
                    acc[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_cur, hb[p][s], s == 0 ? bias : acc[p], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                a_cur = a_nxt;
            }
            const bf16x8_t f0 = hf[(2 * mt) * 64], f1 = hf[(2 * mt + 1) * 64];
#pragma unroll
            for (int p = 0; p < PT; ++p) {
                hd[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f0, relu_pack(acc[p], 0), hd[p], 0, 0, 0);
                hd[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f1, relu_pack(acc[p], 1), hd[p], 0, 0, 0);
            }
        }
#pragma unroll
        for (int p = 0; p < PT; ++p) {
            if (h == 0 && valid[p]) {
                const int64_t q = r[p] * A.N + i[p];
                A.scores[q] = hd[p][0];
                A.errb[q] = A.band_rel * (hd[p][1] + fabsf(b3));
            }
        }
    }
}

bool mfma_supported(const ModelDims& m) {
    return m.bf16 && m.L == 2 && (m.d == 16 || m.d == 32 || m.d == 48 || m.d == 64) &&
           (m.h1 == 64 || m.h1 == 128 || m.h1 == 256) && m.h1 == m.h2;
}

template <int MT>
static void launch_mfma_d(const MfmaArgs& a, int d, int64_t grid, hipStream_t s) {
    if (d == 64) hipLaunchKernelGGL((score_pairs_mfma_kernel<MT, MT, 64>), dim3((uint32_t)grid), dim3(512), 0, s, a);
    else if (d == 48) hipLaunchKernelGGL((score_pairs_mfma_kernel<MT, MT, 48>), dim3((uint32_t)grid), dim3(512), 0, s, a);
    else if (d == 32) hipLaunchKernelGGL((score_pairs_mfma_kernel<MT, MT, 32>), dim3((uint32_t)grid), dim3(512), 0, s, a);
    else hipLaunchKernelGGL((score_pairs_mfma_kernel<MT, MT, 16>), dim3((uint32_t)grid), dim3(512), 0, s, a);
}

hipError_t launch_score_pairs_mfma(const ModelDims& m, const uint16_t* frag16, const float* frag32,
                                   const float* compute, const uint16_t* xinst, const float* mu,
                                   const float* inv_sigma, int32_t R, int32_t N, const int64_t* req_off,
                                   const int32_t* prompt_len, const int32_t* overlap, float* scores, float* errb,
                                   int n_cu, hipStream_t s) {
    const MfmaLayout Lay = make_mfma_layout(m);
    MfmaArgs a;
    a.w1frag = reinterpret_cast<const bf16x8_t*>(frag16);
    a.w2frag = reinterpret_cast<const bf16x8_t*>(frag16 + Lay.w1_frags * 512);
    a.hfrag = reinterpret_cast<const bf16x8_t*>(frag16 + (Lay.w1_frags + Lay.w2_frags) * 512);
    a.b1frag = frag32;
    a.b2frag = frag32 + (m.h1 / 32) * 32;
    a.b3 = compute + m.c_b3;
    a.xinst = xinst;
    a.mu = mu;
    a.isig = inv_sigma;
    a.req_off = req_off;
    a.prompt_len = prompt_len;
    a.overlap = overlap;
    a.scores = scores;
    a.errb = errb;
    a.R = R;
    a.N = N;
    a.d = m.d;
    a.d_inst = m.d_inst;
    a.block_tokens = m.block_tokens;
    a.band_rel = kBandRel;
    const int64_t tiles = (int64_t)R * ((N + 31) / 32);
    int64_t grid = (tiles + 15) / 16;                      // 8 waves of 2 tiles
    if (grid > n_cu) grid = n_cu;
    if (grid < 1) grid = 1;
    if (m.h1 == 256) launch_mfma_d<8>(a, m.d, grid, s);
    else if (m.h1 == 128) launch_mfma_d<4>(a, m.d, grid, s);
    else launch_mfma_d<2>(a, m.d, grid, s);
    return hipGetLastError();
}

}  // namespace ls
