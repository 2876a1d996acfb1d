// K4: one online SGD step of the reward model.
//
// The paper retrains the predictor online from logged (features, observed
// TTFT) records (Section 4.3.2) but states neither loss nor optimiser; this
// library takes the mean squared error of the TTFT prediction and plain SGD:
//   L = (1/B) sum_b (t_b - y_b)^2,   W <- W - lr * dL/dW.
// Forward activations are saved feature-major ([unit][sample]) so every kernel
// reads them coalesced; weight gradients are K = B reductions done as split-K
// tiles with a fixed partition and a fixed-order second pass, so a step is
// bitwise reproducible.  In bf16 mode every multiplication operand (weights,
// layer inputs, each layer's output gradient) is a bf16 value; sums are fp32.
#include <algorithm>
#include <type_traits>

#include "k_policy.h"

namespace ls {

__device__ __forceinline__ float q_bf16(float x) {
    if (x != x) return x;
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

__device__ __forceinline__ float relu_u(float z) { return z > 0.0f ? z : 0.0f; }

// Dropout of unit j of hidden layer `layer` for row b (see DropArgs).
__device__ __forceinline__ bool drop_unit(const DropArgs& D, int layer, int64_t b, int j) {
    const uint64_t c = ((((D.step * 4u + (uint64_t)layer) << 24) | (uint64_t)b) << 10) | (uint64_t)j;
    return (mix64(D.seed + (c + 1u) * 0x9e3779b97f4a7c15ull) >> 11) < D.thr53;
}

// A hidden activation after dropout (before any bf16 rounding), and likewise a
// hidden unit's gradient: 0 if dropped, times the scale if kept.
__device__ __forceinline__ float apply_drop(const DropArgs& D, int layer, int64_t b, int j, float v) {
    if (D.thr53 == 0) return v;
    return drop_unit(D, layer, b, j) ? 0.0f : __fmul_rn(v, D.scale);
}

static inline uint32_t blocks_for(int64_t n, int block) { return (uint32_t)((n + block - 1) / block); }

// Storage of the update's saved activations and layer gradients: fp32, or, for
// bf16 models whose layers all run on the matrix cores, the bf16 bit patterns
// (every stored value is already a bf16 number there, so nothing is lost and
// each pass moves half the bytes).
typedef uint16_t bf16s_t;
__device__ __forceinline__ float ld_act(const float* __restrict__ p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_act(const bf16s_t* __restrict__ p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}
__device__ __forceinline__ void st_act(float* __restrict__ p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void st_act(bf16s_t* __restrict__ p, int64_t i, float v) {
    p[i] = v != v ? (bf16s_t)0x7FC0u : (bf16s_t)(__float_as_uint(v) >> 16);
}

// ---------------------------------------------------------------------------
// workspace layout
// ---------------------------------------------------------------------------
struct UpdWs {
    float *xn, *t, *g, *grad, *part, *loss_part;
    uint64_t* zb[3];                 // per hidden layer: ReLU mask (z > 0), one bit per sample
    float *a[3], *dl[3];             // per hidden layer: activation, dL/dz
    int64_t bytes;
    int S;              // split-K chunks
    int64_t chunk;      // samples per chunk (multiple of 16)
    int loss_blocks;
};

constexpr int kWgradChunk = 512;     // samples per split-K chunk (multiple of 16)
constexpr int kWgradMaxChunks = 256;

struct WgradPlan {
    int S;
    int64_t chunk;
};

// Chunks of 512 samples (of 64 for a single m-tile, whose partials are tiny).
static WgradPlan wgrad_plan(int32_t B, int M) {
    const int64_t c0 = M <= 32 ? 64 : kWgradChunk;
    const int64_t cap = M <= 32 ? 4 * kWgradMaxChunks : kWgradMaxChunks;
    int64_t S = ((int64_t)B + c0 - 1) / c0;
    if (S < 1) S = 1;
    if (S > cap) S = cap;
    int64_t chunk = ((int64_t)B + S - 1) / S;
    chunk = (chunk + 63) & ~int64_t(63);
    S = ((int64_t)B + chunk - 1) / chunk;
    if (S < 1) S = 1;
    return {(int)S, chunk};
}

static int64_t align_floats(int64_t n) { return (n + 63) & ~int64_t(63); }

static UpdWs plan_ws(const ModelDims& m, int32_t B, char* base) {
    UpdWs w{};
    // vector-ALU weight gradients: chunks of 64 samples (up to 256 chunks), so
    // that even a one-row gradient spreads over many workgroups; the partition
    // depends on B alone, so the summation order is fixed
    int64_t S0 = ((int64_t)B + 63) / 64;
    int S = (int)(S0 < 1 ? 1 : (S0 > 256 ? 256 : S0));
    int64_t chunk = ((int64_t)B + S - 1) / S;
    chunk = (chunk + 15) & ~int64_t(15);
    S = (int)(((int64_t)B + chunk - 1) / chunk);
    w.S = S;
    w.chunk = chunk;
    w.loss_blocks = (int)blocks_for(B, 256);
    int64_t maxmn = 0, mfma_floats = 0;
    for (int l = 0; l <= m.L; ++l) {
        const int64_t O = m.out_of(l), K = m.in_of(l);
        maxmn = std::max(maxmn, O * K);
        // the matrix-core weight gradients keep one more column (the bias) per partial
        mfma_floats = std::max(mfma_floats, (int64_t)wgrad_plan(B, (int)O).S * O * (K + 1));
    }
    const int64_t part_floats = std::max<int64_t>((int64_t)S * maxmn, mfma_floats);
    int64_t off = 0;
    auto take = [&](int64_t n) -> float* {
        float* p = base ? reinterpret_cast<float*>(base) + off : nullptr;
        off += align_floats(n);
        return p;
    };
    w.xn = take((int64_t)m.d * B);
    for (int l = 0; l < 3; ++l) {
        const int64_t n = l < m.L ? (int64_t)m.h[l] * B : 0;
        w.zb[l] = l < m.L ? reinterpret_cast<uint64_t*>(take(2 * (int64_t)m.h[l] * ((B + 63) / 64))) : nullptr;
        w.a[l] = l < m.L ? take(n) : nullptr;
        w.dl[l] = l < m.L ? take(n) : nullptr;
    }
    w.t = take(B);
    w.g = take(B);
    w.grad = take(m.n_params);
    w.part = take(part_floats);
    w.loss_part = take(w.loss_blocks);
    w.bytes = off * (int64_t)sizeof(float);
    return w;
}

int64_t update_workspace_bytes(const ModelDims& m, int32_t B) { return plan_ws(m, B, nullptr).bytes; }

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
// Normalised inputs, feature-major: a tile of 64 samples x 64 features is read
// row by row (coalesced), transposed through LDS and written out one feature
// row at a time.
template <bool BF, typename TA = float>
__global__ __launch_bounds__(256) void normalize_kernel(const float* __restrict__ feats, const float* __restrict__ mu,
                                                        const float* __restrict__ isig, TA* __restrict__ xn,
                                                        int32_t B, int d) {
    __shared__ float tile[64][65];                  // [feature][sample]
    const int64_t b0 = (int64_t)blockIdx.x * 64;
    const int c0 = (int)blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int64_t b = b0 + i;
        const int c = c0 + tx;
        float v = 0.0f;
        if (b < B && c < d) v = __fmul_rn(__fsub_rn(feats[b * d + c], mu[c]), isig[c]);
        tile[tx][i] = BF ? q_bf16(v) : v;
    }
    __syncthreads();
    for (int j = ty; j < 64; j += 4) {
        const int c = c0 + j;
        const int64_t b = b0 + tx;
        if (c < d && b < B) st_act(xn, (int64_t)c * B + b, tile[j][tx]);
    }
}

// bf16 storage with B a multiple of 8: the same tiles, written as 16-byte runs
// of eight consecutive samples of a feature row.  Same values as
// normalize_kernel.
__global__ __launch_bounds__(256) void normalize_b16_kernel(const float* __restrict__ feats,
                                                            const float* __restrict__ mu,
                                                            const float* __restrict__ isig, bf16s_t* __restrict__ xn,
                                                            int32_t B, int d) {
    __shared__ float tile[64][65];                  // [feature][sample]
    const int64_t b0 = (int64_t)blockIdx.x * 64;
    const int c0 = (int)blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int c = c0 + tx;
    const float m_c = c < d ? mu[c] : 0.0f, s_c = c < d ? isig[c] : 0.0f;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        const int i = ty + 4 * q;
        const int64_t b = b0 + i;
        float v = 0.0f;
        if (b < B && c < d) v = __fmul_rn(__fsub_rn(feats[b * d + c], m_c), s_c);
        tile[tx][i] = q_bf16(v);
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int p = (int)threadIdx.x + 256 * q;
        const int j = p >> 3, s8 = (p & 7) * 8;
        const int cj = c0 + j;
        const int64_t b = b0 + s8;
        if (cj >= d || b >= B) continue;            // b + 8 <= B: B and b are multiples of 8
        bf16s_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) st_act(h, e, tile[j][s8 + e]);
        uint4 pk;
        pk.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
        pk.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
        pk.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
        pk.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
        *reinterpret_cast<uint4*>(xn + (int64_t)cj * B + b) = pk;
    }
}

// ReLU masks of the hidden layers: the backward pass only needs z > 0 of each
// pre-activation, so the forward keeps one bit per (unit, sample), bit b & 63
// of word o * ceil(B / 64) + (b >> 6), instead of z itself (2 MB instead of
// 67 MB per 256-unit layer at B = 65,536).  A wave of 64 consecutive samples
// writes a whole word with one ballot.
__host__ __device__ __forceinline__ int64_t mask_words(int32_t B) { return ((int64_t)B + 63) >> 6; }
__device__ __forceinline__ bool mask_bit(const uint64_t* __restrict__ zb, int32_t B, int o, int64_t b) {
    return (zb[(int64_t)o * mask_words(B) + (b >> 6)] >> (b & 63)) & 1ull;
}

// U consecutive output units of one sample: each is the fma chain from its bias
// over the inputs in ascending order.  Inputs are fetched eight at a time ahead
// of their multiply-adds; the order of every chain is unchanged.
template <bool BF, bool RELU, int U>
__device__ __forceinline__ void fwd_units(const float* __restrict__ in, const float* __restrict__ wt,
                                          const float* __restrict__ bias, float* __restrict__ z,
                                          uint64_t* __restrict__ zb, float* __restrict__ a, int32_t B, int K, int O,
                                          int jb, int64_t b, int64_t wsamp, bool valid, const DropArgs& D, int layer) {
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = bias[jb + u];
    int k = 0;
    for (; k + 8 <= K; k += 8) {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = in[(int64_t)(k + e) * B + b];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float* __restrict__ w = wt + (int64_t)(k + e) * O + jb;
#pragma unroll
            for (int u = 0; u < U; ++u) acc[u] = __builtin_fmaf(w[u], x[e], acc[u]);
        }
    }
    for (; k < K; ++k) {
        const float x = in[(int64_t)k * B + b];
        const float* __restrict__ w = wt + (int64_t)k * O + jb;
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] = __builtin_fmaf(w[u], x, acc[u]);
    }
    if (RELU && zb != nullptr) {                     // uniform; the wave's samples start at wsamp
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t mk = __ballot(valid && acc[u] > 0.0f);
            if ((threadIdx.x & 63) == 0 && wsamp < B) zb[(int64_t)(jb + u) * mask_words(B) + (wsamp >> 6)] = mk;
        }
    }
    if (!valid) return;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (RELU) {
            const float h = apply_drop(D, layer, b, jb + u, relu_u(acc[u]));
            a[(int64_t)(jb + u) * B + b] = BF ? q_bf16(h) : h;
        } else {
            z[(int64_t)(jb + u) * B + b] = acc[u];
        }
    }
}

// One layer: lane = sample, blockIdx.y = a block of 32 output units (weights
// are uniform across the wave), so a layer runs as (B / 256) x (O / 32)
// workgroups.
template <bool BF, bool RELU>
__global__ __launch_bounds__(256) void layer_fwd_kernel(const float* __restrict__ in, const float* __restrict__ wt,
                                                        const float* __restrict__ bias, float* __restrict__ z,
                                                        uint64_t* __restrict__ zb, float* __restrict__ a, int32_t B,
                                                        int K, int O, DropArgs D, int layer) {
    int64_t bt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t wsamp = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~63u);
    bool valid = bt < B;
    int64_t b = valid ? bt : 0;
    int jb = blockIdx.y * 32;
    const int rem = O - jb;
    if (rem >= 32) { fwd_units<BF, RELU, 32>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); return; }
    if (rem & 16) { fwd_units<BF, RELU, 16>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); jb += 16; }
    if (rem & 8) { fwd_units<BF, RELU, 8>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); jb += 8; }
    if (rem & 4) { fwd_units<BF, RELU, 4>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); jb += 4; }
    if (rem & 2) { fwd_units<BF, RELU, 2>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); jb += 2; }
    if (rem & 1) { fwd_units<BF, RELU, 1>(in, wt, bias, z, zb, a, B, K, O, jb, b, wsamp, valid, D, layer); jb += 1; }
}

// The same chains with the weights of the workgroup's 32 output units staged
// in LDS (wl[k][u], read as broadcasts) instead of fetched per wave.  One
// kernel serves the three lane-per-sample products of the step:
//   kFwdRelu   z = b + W a, a' = relu(z) (bf16 in bf16 mode); weight(k, o) = wt[k][o]
//   kFwdHead   t = b3 + w3 . a2 (one output);                  weight(k, o) = wt[k][o]
//   kBackprop  d1 = [z1 > 0] (W2^T d2) (bf16 in bf16 mode), the chain starting
//              from zero;                                        weight(k, o) = wt[o][k]
// where wt is the compute copy's W1T, W2T or w3.  Every chain keeps its order:
// bias (or zero) first, then inputs k ascending.
constexpr int kDenseMaxK = 256;
enum DenseMode { kFwdRelu = 0, kFwdHead = 1, kBackprop = 2 };

// Each lane carries kDenseSpl samples (64 apart), so one LDS weight read feeds
// kDenseSpl chains, and a workgroup covers kDenseUnits output units.  The
// weights reach the lanes as LDS broadcasts: a 16-byte read returns 1 KiB to
// the wave, about 8 cycles of the compute unit's LDS, and feeds 4 kDenseSpl
// fma instructions of 4 cycles on one SIMD, so four samples per lane keep the
// LDS at half the rate the four SIMDs' fmas need (two samples saturate it).
constexpr int kDenseSpl = 4;
constexpr int kDenseUnits = 16;

// The end of one chain of the three products above: sample b, output unit o,
// element e = o * B + b of the feature-major outputs.
// `on` is the ReLU mask bit of (o, b) in kBackprop.
template <bool BF, int MODE>
__device__ __forceinline__ void dense_store(float acc, int64_t e, int64_t b, int o, bool on, float* __restrict__ z,
                                            float* __restrict__ a, const DropArgs& D, int layer) {
    if (MODE == kFwdRelu) {
        const float h = apply_drop(D, layer, b, o, relu_u(acc));
        a[e] = BF ? q_bf16(h) : h;
    } else if (MODE == kFwdHead) {
        z[e] = acc;
    } else {
        const float v = apply_drop(D, layer, b, o, on ? acc : 0.0f);
        z[e] = BF ? q_bf16(v) : v;
    }
}

// The value dense_store stores, for kernels that store it themselves.
template <bool BF, int MODE>
__device__ __forceinline__ float dense_value(float acc, int64_t b, int o, bool on, const DropArgs& D, int layer) {
    float v;
    if (MODE == kFwdRelu) v = apply_drop(D, layer, b, o, relu_u(acc));
    else if (MODE == kFwdHead) return acc;
    else v = apply_drop(D, layer, b, o, on ? acc : 0.0f);
    return BF ? q_bf16(v) : v;
}

// zb: the layer's ReLU mask, written in kFwdRelu (when not null) and read in
// kBackprop; wsamp: the wave's first sample (slot j holds wsamp + 64 j + lane).
template <bool BF, int MODE, int U>
__device__ __forceinline__ void dense_units(const float* __restrict__ in, const float* __restrict__ wl,
                                            const float* __restrict__ bias, uint64_t* __restrict__ zb,
                                            float* __restrict__ z, float* __restrict__ a, int32_t B, int K, int o0,
                                            int uoff, const int64_t (&b)[kDenseSpl], const bool (&valid)[kDenseSpl],
                                            int64_t wsamp, const DropArgs& D, int layer) {
    constexpr int P = kDenseSpl;
    float acc[P][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float init = MODE == kBackprop ? 0.0f : bias[o0 + u];
#pragma unroll
        for (int j = 0; j < P; ++j) acc[j][u] = init;
    }
    int k = 0;
    for (; k + 4 <= K; k += 4) {
        float x[4][P];
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int j = 0; j < P; ++j) x[e][j] = in[(int64_t)(k + e) * B + b[j]];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float* __restrict__ w = wl + (k + e) * kDenseUnits + uoff;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float wv = w[u];
#pragma unroll
                for (int j = 0; j < P; ++j) acc[j][u] = __builtin_fmaf(wv, x[e][j], acc[j][u]);
            }
        }
    }
    for (; k < K; ++k) {
        const float* __restrict__ w = wl + k * kDenseUnits + uoff;
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const float x = in[(int64_t)k * B + b[j]];
#pragma unroll
            for (int u = 0; u < U; ++u) acc[j][u] = __builtin_fmaf(w[u], x, acc[j][u]);
        }
    }
#pragma unroll
    for (int j = 0; j < P; ++j) {
        const int64_t ws = wsamp + 64 * j;
        if (MODE == kFwdRelu && zb != nullptr) {         // uniform
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint64_t mk = __ballot(valid[j] && acc[j][u] > 0.0f);
                if ((threadIdx.x & 63) == 0 && ws < B) zb[(int64_t)(o0 + u) * mask_words(B) + (ws >> 6)] = mk;
            }
        }
        if (!valid[j]) continue;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            bool on = true;
            if (MODE == kBackprop) on = mask_bit(zb, B, o0 + u, b[j]);
            dense_store<BF, MODE>(acc[j][u], (int64_t)(o0 + u) * B + b[j], b[j], o0 + u, on, z, a, D, layer);
        }
    }
}

// Four waves per SIMD (at most 128 VGPRs): at the Large update's 1,024
// workgroups every one is resident at once.
template <bool BF, int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void dense_lane_kernel(
    const float* __restrict__ in, const float* __restrict__ wt,
                                                         const float* __restrict__ bias,
                                                         uint64_t* __restrict__ zb, float* __restrict__ z,
                                                         float* __restrict__ a, int32_t B, int K, int O, DropArgs D,
                                                         int layer) {
    __shared__ __align__(16) float wl[kDenseMaxK * kDenseUnits];
    const int jb = blockIdx.y * kDenseUnits;
    const int nu = O - jb < kDenseUnits ? O - jb : kDenseUnits;
    lds_fill<8>(wl, K * kDenseUnits, [&](int e) {
        const int k = e / kDenseUnits, u = e % kDenseUnits;
        float v = 0.0f;
        if (u < nu) v = MODE == kBackprop ? wt[(int64_t)(jb + u) * K + k] : wt[(int64_t)k * O + jb + u];
        return v;
    });
    __syncthreads();
    // samples of this lane: block base + wave * 64 P + 64 j + lane
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t wsamp = (int64_t)blockIdx.x * blockDim.x * kDenseSpl + (int64_t)wave * 64 * kDenseSpl;
    const int64_t base = wsamp + lane;
    int64_t b[kDenseSpl];
    bool valid[kDenseSpl];
#pragma unroll
    for (int j = 0; j < kDenseSpl; ++j) {
        const int64_t bt = base + 64 * j;
        valid[j] = bt < B;
        b[j] = valid[j] ? bt : 0;
    }
    if (nu == kDenseUnits) {
        dense_units<BF, MODE, kDenseUnits>(in, wl, bias, zb, z, a, B, K, jb, 0, b, valid, wsamp, D, layer);
        return;
    }
    static_assert(kDenseUnits <= 32 && (kDenseUnits & (kDenseUnits - 1)) == 0, "a power of two up to 32");
    int uo = 0;
    if (kDenseUnits > 16 && (nu & 16)) { dense_units<BF, MODE, 16>(in, wl, bias, zb, z, a, B, K, jb + uo, uo, b, valid, wsamp, D, layer); uo += 16; }
    if (nu & 8) { dense_units<BF, MODE, 8>(in, wl, bias, zb, z, a, B, K, jb + uo, uo, b, valid, wsamp, D, layer); uo += 8; }
    if (nu & 4) { dense_units<BF, MODE, 4>(in, wl, bias, zb, z, a, B, K, jb + uo, uo, b, valid, wsamp, D, layer); uo += 4; }
    if (nu & 2) { dense_units<BF, MODE, 2>(in, wl, bias, zb, z, a, B, K, jb + uo, uo, b, valid, wsamp, D, layer); uo += 2; }
    if (nu & 1) { dense_units<BF, MODE, 1>(in, wl, bias, zb, z, a, B, K, jb + uo, uo, b, valid, wsamp, D, layer); uo += 1; }
}

// The same products for small batches, where a workgroup per 32 output units
// and 512 samples leaves most CUs idle: one thread per (sample, output unit),
// 64 units by 4 samples per workgroup (the head, one unit: 256 samples), the
// weights read from the compute copy (L2-resident) and the inputs as
// wave-uniform loads.  Same chains, same order.
constexpr int kDenseSmallWgs = 256;            // below this many lane-path workgroups

template <bool BF, int MODE, typename TIN = float>
__global__ __launch_bounds__(256) void dense_small_kernel(const TIN* __restrict__ in, const float* __restrict__ wt,
                                                          const float* __restrict__ bias,
                                                          uint64_t* __restrict__ zb, float* __restrict__ z,
                                                          float* __restrict__ a, int32_t B, int K, int O, DropArgs D,
                                                          int layer) {
    const int o = MODE == kFwdHead ? 0 : (int)blockIdx.x * 64 + (int)(threadIdx.x & 63);
    const int64_t b = MODE == kFwdHead ? (int64_t)blockIdx.y * 256 + threadIdx.x
                                       : (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6);
    if (o >= O || b >= B) return;
    float acc = MODE == kBackprop ? 0.0f : bias[o];
    int k = 0;
    for (; k + 8 <= K; k += 8) {
        float w[8], x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            w[e] = MODE == kBackprop ? wt[(int64_t)o * K + k + e] : wt[(int64_t)(k + e) * O + o];
            x[e] = ld_act(in, (int64_t)(k + e) * B + b);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = __builtin_fmaf(w[e], x[e], acc);
    }
    for (; k < K; ++k) {
        const float w = MODE == kBackprop ? wt[(int64_t)o * K + k] : wt[(int64_t)k * O + o];
        acc = __builtin_fmaf(w, ld_act(in, (int64_t)k * B + b), acc);
    }
    // the mask bits of a word come from different threads here: zb starts zeroed
    if (MODE == kFwdRelu && zb != nullptr && acc > 0.0f)
        atomicOr(reinterpret_cast<unsigned long long*>(zb + (int64_t)o * mask_words(B) + (b >> 6)), 1ull << (b & 63));
    const bool on = MODE == kBackprop ? mask_bit(zb, B, o, b) : true;
    dense_store<BF, MODE>(acc, (int64_t)o * B + b, b, o, on, z, a, D, layer);
}

static bool dense_small(int32_t B, int O) {
    return (int64_t)((B + 256 * kDenseSpl - 1) / (256 * kDenseSpl)) * ((O + kDenseUnits - 1) / kDenseUnits) <
           kDenseSmallWgs;
}

// The same chains on the matrix cores.  v_mfma_f32_32x32x1_2b_f32 gives each
// of its outputs one multiply-add rounded once, as fmaf does (denormals kept),
// so an accumulator that starts at the bias and takes the inputs k = 0, 1, ...
// one instruction each holds the chain's value bit for bit.  A wave owns 64
// samples (block 0: the first 32, block 1: the next 32) and kMfTiles tiles of
// 32 output units; per input k its B operand is row k of the feature-major
// input, one coalesced 256-byte load, and each tile's A operand is the unit
// slice's weight column k.  The accumulator's rows are units: register i of
// lane l holds unit 8 (i % 16 / 4) + 4 (l / 32) + i % 4 of its tile, sample
// 32 (i / 16) + l % 32 of the wave.
//
// The slice sits in LDS unit-major, wl[u][k] with a row stride of mf_ldk(K)
// floats (K rounded up to 4, plus 4 when that is a multiple of 8), so that one
// 16-byte read gives a lane its unit's weights for four consecutive k and the
// 32 lanes of a tile read without bank conflicts.  A group of kMfPre inputs
// takes all of its A operands in one batch of reads issued before its first
// multiply-add, and its B operands one group ahead.
constexpr int kMfWaves = 8;                   // 64 samples each
constexpr int kMfPre = 8;                     // inputs per group
constexpr int kMfMaxLdk = kDenseMaxK + 4;

__host__ __device__ constexpr int mf_ldk(int K) {
    return ((K + 3) & ~3) + ((((K + 3) >> 2) & 1) ? 0 : 4);
}

typedef float f32x32_t __attribute__((ext_vector_type(32)));

// DROP: dropout on (the stores then draw each unit's mask).  A wave whose 64
// samples and 128 units all exist (every wave but the edges) takes the
// epilogue without per-element tests: row bases are scalar, lane offsets 32-bit,
// and the ReLU mask words of its 128 units are gathered into two registers per
// lane and written with two stores.
template <bool BF, int MODE, bool DROP, int TILES, typename TA = float>
__global__ __launch_bounds__(64 * kMfWaves) void dense_mfma_kernel(const TA* __restrict__ in,
                                                                   const float* __restrict__ wt,
                                                                   const float* __restrict__ bias,
                                                                   uint64_t* __restrict__ zb, TA* __restrict__ z,
                                                                   TA* __restrict__ a, int32_t B, int K, int O,
                                                                   DropArgs D, int layer) {
    static_assert(MODE == kFwdRelu || MODE == kBackprop, "hidden layers only");
    static_assert(TILES == 1 || TILES == 2 || TILES == 4, "tiles per wave");
    constexpr int kMfUnits = 32 * TILES;          // output units per workgroup
    constexpr int kMfTiles = TILES;
    constexpr int NW = (kMfUnits + 63) / 64;      // mask-word registers per lane
    __shared__ __align__(16) float wl[kMfUnits * kMfMaxLdk];
    __shared__ __align__(16) float bl[kMfUnits];
    const int jb = blockIdx.y * kMfUnits;
    const int nu = O - jb < kMfUnits ? O - jb : kMfUnits;
    const int ldk = mf_ldk(K);
    const int tid = (int)threadIdx.x, T_ = (int)blockDim.x;
    // the slice, zero past O and past K
    if ((MODE == kBackprop ? (K & 3) == 0 : (O & 3) == 0) && (reinterpret_cast<uintptr_t>(wt) & 15) == 0) {
        // 16-byte loads, all of a thread's in flight at once.  Gradients (wt is
        // [units][K]): a load is four k of one unit, written as one 16-byte LDS
        // store.  Forward (wt is [K][O]): a load is four units of one k; a wave's
        // 64 loads cover 16 units x 16 k (64-byte runs of wt), so that its four
        // 4-byte LDS stores each hit 64 distinct banks (row stride = 4 mod 64).
        constexpr int kFillMax = (kMfUnits * kMfMaxLdk / 4 + 64 * kMfWaves - 1) / (64 * kMfWaves) + 1;
        const int q4 = ldk >> 2;
        const int n4 = MODE == kBackprop ? kMfUnits * q4 : (kMfUnits / 16) * ((ldk + 15) >> 4) * 64;
        float4 v[kFillMax];
        bool ok[kFillMax];            // zeroed at the LDS write: no register write behind a pending load
        auto where = [&](int e, int& u, int& k) {
            if (MODE == kBackprop) {
                u = e / q4;
                k = 4 * (e - u * q4);
            } else {
                const int tile = e >> 6, l = e & 63;
                k = 16 * (tile / (kMfUnits / 16)) + (l >> 2);
                u = 16 * (tile % (kMfUnits / 16)) + 4 * (l & 3);
            }
        };
#pragma unroll
        for (int j = 0; j < kFillMax; ++j) {
            const int e = tid + j * T_ < n4 ? tid + j * T_ : n4 - 1;
            int u, k;
            where(e, u, k);
            // clamped into the slice: a whole float4 of units (forward) or of k (gradients)
            const int uc = u < nu ? u : (MODE == kBackprop ? nu - 1 : nu - 4);
            const int kc = k < K ? k : (MODE == kBackprop ? K - 4 : K - 1);
            v[j] = MODE == kBackprop ? *reinterpret_cast<const float4*>(wt + (int64_t)(jb + uc) * K + kc)
                                     : *reinterpret_cast<const float4*>(wt + (int64_t)kc * O + jb + uc);
            ok[j] = u < nu && k < K;
        }
#pragma unroll
        for (int j = 0; j < kFillMax; ++j) {
            const int e = tid + j * T_;
            if (e >= n4) break;
            int u, k;
            where(e, u, k);
            if (k >= ldk) continue;
            const float4 q = ok[j] ? v[j] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (MODE == kBackprop) {
                *reinterpret_cast<float4*>(wl + u * ldk + k) = q;
            } else {
                wl[(u + 0) * ldk + k] = q.x;
                wl[(u + 1) * ldk + k] = q.y;
                wl[(u + 2) * ldk + k] = q.z;
                wl[(u + 3) * ldk + k] = q.w;
            }
        }
    } else {
        const int n = kMfUnits * ldk;
        for (int e0 = tid; e0 < n; e0 += 16 * T_) {
            float v[16];
            bool ok[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int e = e0 + j * T_ < n ? e0 + j * T_ : n - 1;
                int k, u;
                if (MODE == kBackprop) {
                    u = e / ldk;
                    k = e - u * ldk;
                } else {
                    k = e / kMfUnits;
                    u = e - k * kMfUnits;
                }
                const int uc = u < nu ? u : nu - 1, kc = k < K ? k : K - 1;
                v[j] = MODE == kBackprop ? wt[(int64_t)(jb + uc) * K + kc] : wt[(int64_t)kc * O + jb + uc];
                ok[j] = u < nu && k < K;
            }
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int e = e0 + j * T_;
                if (e < n) {
                    int k, u;
                    if (MODE == kBackprop) {
                        u = e / ldk;
                        k = e - u * ldk;
                    } else {
                        k = e / kMfUnits;
                        u = e - k * kMfUnits;
                    }
                    wl[u * ldk + k] = ok[j] ? v[j] : 0.0f;
                }
            }
        }
    }
    if (tid < kMfUnits) bl[tid] = (MODE == kBackprop || tid >= nu) ? 0.0f : bias[jb + tid];
    __syncthreads();
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t b0 = (int64_t)blockIdx.x * (64 * kMfWaves) + 64 * wave;
    if (b0 >= B) return;
    const int64_t bl_ = b0 + lane;
    const TA* __restrict__ src = in + (bl_ < B ? bl_ : (int64_t)B - 1);      // lanes past B read a valid row
    const int hi = lane >> 5, col = lane & 31;
    // accumulators start at the bias (zero for the gradients and for units past O)
    f32x32_t acc[kMfTiles];
#pragma unroll
    for (int t = 0; t < kMfTiles; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float4 q = *reinterpret_cast<const float4*>(bl + 32 * t + 8 * r + 4 * hi);
            acc[t][4 * r + 0] = acc[t][16 + 4 * r + 0] = q.x;
            acc[t][4 * r + 1] = acc[t][16 + 4 * r + 1] = q.y;
            acc[t][4 * r + 2] = acc[t][16 + 4 * r + 2] = q.z;
            acc[t][4 * r + 3] = acc[t][16 + 4 * r + 3] = q.w;
        }
    // tile t's unit for this lane: row (32 t + col) of the slice
    const float* __restrict__ wrow = wl + col * ldk;
    // inputs k0 .. k0 + kMfPre - 1 (rows past K clamped to K - 1: always in bounds)
    auto load = [&](float (&x)[kMfPre], int k0) {
#pragma unroll
        for (int e = 0; e < kMfPre; ++e) {
            const int k = k0 + e < K ? k0 + e : K - 1;
            x[e] = ld_act(src, (int64_t)k * B);
        }
    };
    // one group of inputs; FULL: all kMfPre of them are below K (no per-step test,
    // so the reads of the A operands stay ahead of the multiply-adds)
    auto step = [&](const float (&x)[kMfPre], int k0, auto full) {
        float4 w[kMfPre / 4][kMfTiles];
#pragma unroll
        for (int g = 0; g < kMfPre / 4; ++g)
#pragma unroll
            for (int t = 0; t < kMfTiles; ++t) {
                const int kk = k0 + 4 * g < ldk - 3 ? k0 + 4 * g : ldk - 4;
                w[g][t] = *reinterpret_cast<const float4*>(wrow + 32 * t * ldk + kk);
            }
#pragma unroll
        for (int e = 0; e < kMfPre; ++e) {
            if (!decltype(full)::value && k0 + e >= K) break;
#pragma unroll
            for (int t = 0; t < kMfTiles; ++t) {
                const float4 q = w[e >> 2][t];
                const float wv = (e & 3) == 0 ? q.x : (e & 3) == 1 ? q.y : (e & 3) == 2 ? q.z : q.w;
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x1f32(wv, x[e], acc[t], 0, 0, 0);
            }
        }
    };
    using Full = std::integral_constant<bool, true>;
    using Tail = std::integral_constant<bool, false>;
    float xa[kMfPre], xb[kMfPre];
    load(xa, 0);
    int k0 = 0;
    for (; k0 + 2 * kMfPre <= K; k0 += 2 * kMfPre) {
        load(xb, k0 + kMfPre);
        step(xa, k0, Full{});
        load(xa, k0 + 2 * kMfPre);
        step(xb, k0 + kMfPre, Full{});
    }
    if (k0 < K) {
        load(xb, k0 + kMfPre);
        step(xa, k0, Tail{});
        if (k0 + kMfPre < K) step(xb, k0 + kMfPre, Tail{});
    }
    // epilogue: masks, ReLU or masked gradient, dropout, bf16 rounding.  Register
    // i of tile t holds unit u = 32 t + 8 (i % 16 / 4) + 4 hi + i % 4 of the slice
    // for sample b0 + 32 (i / 16) + col.
    const int mw = (int)mask_words(B);
    TA* __restrict__ outp = MODE == kFwdRelu ? a : z;
    if (b0 + 64 <= B && nu == kMfUnits) {
        // mask words of this wave's sample word for units lane and 64 + lane
        uint32_t wlo[NW], whi[NW];
#pragma unroll
        for (int h = 0; h < NW; ++h) wlo[h] = whi[h] = 0u;
        if (MODE == kBackprop) {
#pragma unroll
            for (int h = 0; h < NW; ++h) {
                const int u = 64 * h + lane < kMfUnits ? 64 * h + lane : kMfUnits - 1;
                const uint64_t w = zb[(int64_t)(jb + u) * mw + (b0 >> 6)];
                wlo[h] = (uint32_t)w;
                whi[h] = (uint32_t)(w >> 32);
            }
        }
        const uint32_t loff = (uint32_t)(4 * hi) * (uint32_t)B + (uint32_t)col;   // lane offset from a row base
#pragma unroll
        for (int t = 0; t < kMfTiles; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int u0 = 32 * t + 8 * (i >> 2) + (i & 3);          // lanes 0-31: u0, lanes 32-63: u0 + 4
                TA* __restrict__ row = outp + (int64_t)(jb + u0) * B + b0;
                float c0 = acc[t][i], c1 = acc[t][i + 16];
                if (MODE == kFwdRelu) {
                    if (zb != nullptr) {     // uniform
                        const uint64_t m0 = __ballot(c0 > 0.0f), m1 = __ballot(c1 > 0.0f);
                        const int h = u0 >> 6, ln = u0 & 63;
                        if (lane == ln) {
                            wlo[h] = (uint32_t)m0;
                            whi[h] = (uint32_t)m1;
                        }
                        if (lane == ln + 4) {
                            wlo[h] = (uint32_t)(m0 >> 32);
                            whi[h] = (uint32_t)(m1 >> 32);
                        }
                    }
                    c0 = relu_u(c0);
                    c1 = relu_u(c1);
                } else {
                    // this lane's unit's word: lane u0 (+ 4) of the gathered words
                    const int h = u0 >> 6, ln = (u0 & 63) + 4 * hi;
                    const uint32_t lo = __builtin_amdgcn_ds_bpermute(ln << 2, (int)wlo[h]);
                    const uint32_t hw = __builtin_amdgcn_ds_bpermute(ln << 2, (int)whi[h]);
                    if (!((lo >> col) & 1u)) c0 = 0.0f;
                    if (!((hw >> col) & 1u)) c1 = 0.0f;
                }
                if (DROP) {
                    const int o = jb + u0 + 4 * hi;
                    c0 = apply_drop(D, layer, b0 + col, o, c0);
                    c1 = apply_drop(D, layer, b0 + 32 + col, o, c1);
                }
                st_act(row, loff, BF ? q_bf16(c0) : c0);
                st_act(row, loff + 32, BF ? q_bf16(c1) : c1);
            }
        if (MODE == kFwdRelu && zb != nullptr) {
#pragma unroll
            for (int h = 0; h < NW; ++h)
                if (64 * h + lane < kMfUnits)
                    zb[(int64_t)(jb + 64 * h + lane) * mw + (b0 >> 6)] = ((uint64_t)whi[h] << 32) | wlo[h];
        }
        return;
    }
    // edge waves: per-element tests
    const int64_t s0 = b0 + col, s1 = b0 + 32 + col;
    const bool v0 = s0 < B, v1 = s1 < B;
#pragma unroll
    for (int t = 0; t < kMfTiles; ++t) {
        const f32x32_t& c = acc[t];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int o = jb + 32 * t + 8 * (i >> 2) + 4 * hi + (i & 3);
            const float c0 = c[i], c1 = c[i + 16];
            bool on0 = true, on1 = true;
            if (MODE == kFwdRelu) {
                if (zb != nullptr) {     // uniform
                    const uint64_t m0 = __ballot(v0 && c0 > 0.0f), m1 = __ballot(v1 && c1 > 0.0f);
                    // lanes 0-31 hold unit o of both blocks, lanes 32-63 unit o + 4
                    const uint64_t word = hi ? ((m0 >> 32) | (m1 & 0xFFFFFFFF00000000ull))
                                             : ((m0 & 0xFFFFFFFFull) | (m1 << 32));
                    if (col == 0 && o < O) zb[(int64_t)o * mw + (b0 >> 6)] = word;
                }
            } else if (o < O) {
                const uint64_t word = zb[(int64_t)o * mw + (b0 >> 6)];
                on0 = (word >> col) & 1ull;
                on1 = (word >> (32 + col)) & 1ull;
            }
            if (o < O) {
                if (v0) st_act(outp, (int64_t)o * B + s0, dense_value<BF, MODE>(c0, s0, o, on0, D, layer));
                if (v1) st_act(outp, (int64_t)o * B + s1, dense_value<BF, MODE>(c1, s1, o, on1, D, layer));
            }
        }
    }
}

// Tiles per wave for the matrix-core chains (0: keep the vector-lane kernels).
// Four (a workgroup per 512 samples and 128 output units) once that fills the
// chip; one (32 units per workgroup, four times the workgroups) for smaller
// batches, down to 16 workgroups; below that the thread-per-element kernels.
constexpr int kMfMinWgs = 128;
constexpr int kMfMinWgs1 = 16;

static int dense_mfma(const ModelDims& m, int32_t B, int O) {
    if (!m.mfma_chains || B > (1 << 28)) return 0;
    const int64_t sb = (B + 64 * kMfWaves - 1) / (64 * kMfWaves);
    if (sb * ((O + 127) / 128) >= kMfMinWgs) return 4;
    if (sb * ((O + 31) / 32) >= kMfMinWgs1) return 1;
    return 0;
}

template <bool BF, int MODE, typename TA = float>
static void launch_dense_mfma(int tiles, const TA* in, const float* wt, const float* bias, uint64_t* zb, TA* z, TA* a,
                              int32_t B, int K, int O, const DropArgs& D, int layer, hipStream_t s) {
    const dim3 block(64 * kMfWaves);
    const dim3 grid(blocks_for(B, 64 * kMfWaves), (O + 32 * tiles - 1) / (32 * tiles));
    if (tiles == 4) {
        if (D.thr53)
            hipLaunchKernelGGL((dense_mfma_kernel<BF, MODE, true, 4, TA>), grid, block, 0, s, in, wt, bias, zb, z, a, B,
                               K, O, D, layer);
        else
            hipLaunchKernelGGL((dense_mfma_kernel<BF, MODE, false, 4, TA>), grid, block, 0, s, in, wt, bias, zb, z, a, B,
                               K, O, D, layer);
    } else {
        if (D.thr53)
            hipLaunchKernelGGL((dense_mfma_kernel<BF, MODE, true, 1, TA>), grid, block, 0, s, in, wt, bias, zb, z, a, B,
                               K, O, D, layer);
        else
            hipLaunchKernelGGL((dense_mfma_kernel<BF, MODE, false, 1, TA>), grid, block, 0, s, in, wt, bias, zb, z, a, B,
                               K, O, D, layer);
    }
}

// ---------------------------------------------------------------------------
// loss and output gradient: g_b = 2 (t_b - y_b) / B
// ---------------------------------------------------------------------------
template <bool BF>
__global__ __launch_bounds__(256) void loss_grad_kernel(const float* __restrict__ t, const float* __restrict__ y,
                                                        float* __restrict__ g, float* __restrict__ loss_part,
                                                        int32_t B) {
    __shared__ float red[256];
    int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    float e2 = 0.0f;
    if (b < B) {
        float err = t[b] - y[b];
        e2 = err * err;
        float gv = (2.0f * err) / (float)B;
        g[b] = BF ? q_bf16(gv) : gv;
    }
    red[threadIdx.x] = e2;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) loss_part[blockIdx.x] = red[0];
}

__global__ void loss_final_kernel(const float* __restrict__ loss_part, int nblk, int32_t B, float* __restrict__ out) {
    __shared__ float red[256];
    float s = 0.0f;
    for (int k = threadIdx.x; k < nblk; k += 256) s += loss_part[k];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = red[0] / (float)B;
}

// dL/dz of the last hidden layer: g_b * w[j] where z > 0 (then dropout's factor);
// blockIdx.y = unit j.  VEC (B a multiple of 4): four consecutive samples per
// thread, one 16-byte load of g and one 16-byte store.
template <bool BF>
__device__ __forceinline__ float head_delta(const float* __restrict__ g, float wj, const uint64_t word, int64_t b,
                                            int j, const DropArgs& D, int layer) {
    const float v = apply_drop(D, layer, b, j, ((word >> (b & 63)) & 1ull) ? g[b] * wj : 0.0f);
    return BF ? q_bf16(v) : v;
}

template <bool BF, bool VEC, typename TA = float>
__global__ __launch_bounds__(256) void delta_head_kernel(const float* __restrict__ g, const float* __restrict__ w,
                                                         const uint64_t* __restrict__ zb, TA* __restrict__ dl,
                                                         int32_t B, DropArgs D, int layer) {
    constexpr int S = VEC ? 4 : 1;
    const int64_t b = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * S;
    const int j = (int)blockIdx.y;
    if (b >= B) return;
    const float wj = w[j];
    const uint64_t word = zb[(int64_t)j * mask_words(B) + (b >> 6)];     // the S samples share it
    const int64_t t = (int64_t)j * B + b;
    if constexpr (VEC && std::is_same<TA, float>::value) {
        *reinterpret_cast<float4*>(dl + t) =
            make_float4(head_delta<BF>(g, wj, word, b, j, D, layer), head_delta<BF>(g, wj, word, b + 1, j, D, layer),
                        head_delta<BF>(g, wj, word, b + 2, j, D, layer), head_delta<BF>(g, wj, word, b + 3, j, D, layer));
    } else if constexpr (VEC) {
        bf16s_t h[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) st_act(h, e, head_delta<BF>(g, wj, word, b + e, j, D, layer));
        uint2 pk;
        pk.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
        pk.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
        *reinterpret_cast<uint2*>(dl + t) = pk;
    } else {
        st_act(dl, t, head_delta<BF>(g, wj, word, b, j, D, layer));
    }
}

// bf16 storage with B a multiple of 8: eight consecutive samples per thread
// (g read once, two 16-byte loads) over kDeltaUnits units (one 16-byte store
// each); blockIdx.y = a group of units.  Same values as delta_head_kernel.
constexpr int kDeltaUnits = 8;

__global__ __launch_bounds__(256) void delta_head_b16_kernel(const float* __restrict__ g, const float* __restrict__ w,
                                                             const uint64_t* __restrict__ zb, bf16s_t* __restrict__ dl,
                                                             int32_t B, int H, DropArgs D, int layer) {
    const int64_t b = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
    if (b >= B) return;                             // b + 8 <= B: B and b are multiples of 8
    const float4 ga = *reinterpret_cast<const float4*>(g + b), gb = *reinterpret_cast<const float4*>(g + b + 4);
    const float gv[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
    const int64_t mw = mask_words(B);
    const int j0 = (int)blockIdx.y * kDeltaUnits;
    // every unit's weight and mask word (the eight samples share it) first
    float wv[kDeltaUnits];
    uint64_t wd[kDeltaUnits];
#pragma unroll
    for (int u = 0; u < kDeltaUnits; ++u) {
        const int j = j0 + u;
        wv[u] = j < H ? w[j] : 0.0f;
        wd[u] = j < H ? zb[(int64_t)j * mw + (b >> 6)] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < kDeltaUnits; ++u) {
        const int j = j0 + u;
        if (j >= H) continue;
        bf16s_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int64_t be = b + e;
            const float v = apply_drop(D, layer, be, j, ((wd[u] >> (be & 63)) & 1ull) ? gv[e] * wv[u] : 0.0f);
            st_act(h, e, q_bf16(v));
        }
        uint4 pk;
        pk.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
        pk.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
        pk.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
        pk.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
        *reinterpret_cast<uint4*>(dl + (int64_t)j * B + b) = pk;
    }
}

// ---------------------------------------------------------------------------
// C_part[s][m][n] = sum_{b in chunk s} A[m][b] * Bt[n][b]   (A [M x B], Bt [N x B])
// 64 x 64 tile per block, 4 x 4 per thread, slabs of 16 samples through LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemm_nt_splitk_kernel(const float* __restrict__ A, const float* __restrict__ Bt,
                                                             float* __restrict__ part, int M, int N, int32_t B,
                                                             int64_t chunk) {
    __shared__ float As[16][64 + 4];
    __shared__ float Bs[16][64 + 4];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
    const int s = blockIdx.z;
    const int64_t kb = (int64_t)s * chunk;
    int64_t ke = kb + chunk;
    if (ke > B) ke = B;
    float acc[4][4] = {};
    const int lrow = tid >> 2, lcol = (tid & 3) * 4;
    for (int64_t k0 = kb; k0 < ke; k0 += 16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int64_t kk = k0 + lcol + e;
            int m = m0 + lrow, n = n0 + lrow;
            As[lcol + e][lrow] = (m < M && kk < ke) ? A[(int64_t)m * B + kk] : 0.0f;
            Bs[lcol + e][lrow] = (n < N && kk < ke) ? Bt[(int64_t)n * B + kk] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
    float* __restrict__ out = part + (int64_t)s * M * N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int m = m0 + ty * 4 + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int n = n0 + tx * 4 + j;
            if (n < N) out[(int64_t)m * N + n] = acc[i][j];
        }
    }
}

// ---------------------------------------------------------------------------
// bf16 mode: weight and bias gradients on the matrix cores.
// C[m][n] = sum_b A[m][b] Bt[n][b] for n < N and C[m][N] = sum_b A[m][b], as
// v_mfma_f32_32x32x16_bf16 with m-tiles as rows, samples as the reduction and
// n-tiles as columns; the bias column comes from one more B operand of ones.
// Every operand is a bf16 value already (layer inputs, output gradients), so
// the products are exact and the sums fp32, as in the VALU path.  Lane l of a
// fragment holds 8 consecutive samples of row l % 32 (samples 8 (l / 32) ..),
// which is exactly 32 contiguous bytes of the feature-major arrays, so the
// operands stream from memory without staging.  Split-K: workgroup s covers a
// fixed chunk of samples; partials are summed in ascending s afterwards.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8_t pack_bf16x8(const float (&v)[8]) {
    // the values are bf16 numbers stored as fp32: the upper halves are exact
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = (__float_as_uint(v[2 * j]) >> 16) | (__float_as_uint(v[2 * j + 1]) & 0xFFFF0000u);
    bf16x8_t out;
    __builtin_memcpy(&out, w, sizeof out);
    return out;
}

// Eight consecutive bf16 values from bf16 storage (VEC: one 16-byte load).
template <bool VEC>
__device__ __forceinline__ bf16x8_t load_frag(const bf16s_t* __restrict__ row, int64_t k, int64_t ke, bool valid) {
    bf16x8_t out;
    if (VEC && valid && k + 8 <= ke) {
        const uint4 p = *reinterpret_cast<const uint4*>(row + k);
        __builtin_memcpy(&out, &p, sizeof out);
    } else {
        uint16_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (valid && k + j < ke) ? row[k + j] : (uint16_t)0;
        __builtin_memcpy(&out, v, sizeof out);
    }
    return out;
}

template <bool VEC>
__device__ __forceinline__ bf16x8_t load_frag(const float* __restrict__ row, int64_t k, int64_t ke, bool valid) {
    float v[8];
    if (VEC && valid && k + 8 <= ke) {
        const float4 p = *reinterpret_cast<const float4*>(row + k);
        const float4 q = *reinterpret_cast<const float4*>(row + k + 4);
        v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w; v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (valid && k + j < ke) ? row[k + j] : 0.0f;
    }
    return pack_bf16x8(v);
}

// One wave per m-tile (eight per workgroup); the B fragments, which every wave
// of the workgroup needs, are converted once into LDS per stage of kWgradKs
// k-steps (double-buffered) and read from there.
constexpr int kWgradKs = 2;

// blockIdx.y = a range of NT n-tiles (the bias column with the first range).
template <int NT, bool VEC, typename TA = float, typename TB = float>
__global__ __launch_bounds__(512) void wgrad_mfma_kernel(const TA* __restrict__ A, const TB* __restrict__ Bt,
                                                         float* __restrict__ part, int M, int N, int32_t B,
                                                         int64_t chunk) {
    const int n0 = (int)blockIdx.y * NT * 32;
    const bool with_bias = blockIdx.y == 0;
    constexpr int KS = kWgradKs;
    constexpr int NE = KS * NT * 64;                 // fragment lanes per stage
    constexpr int EPT = (NE + 511) / 512;            // per thread
    __shared__ bf16x8_t lds_b[2][NE];
    const int tid = threadIdx.x;
    const int lane = tid & 63, mt = tid >> 6;
    const int row = lane & 31, half = lane >> 5;
    const int s = blockIdx.x;
    const int64_t kb = (int64_t)s * chunk;
    const int64_t ke = min(kb + chunk, (int64_t)B);
    const int m = mt * 32 + row;
    const bool mvalid = m < M;
    const TA* __restrict__ arow = A + (int64_t)(mvalid ? m : 0) * B;
    // the fragment lanes this thread stages: (k-step, n-tile, lane) = f
    const TB* __restrict__ srow[EPT];
    bool sval[EPT];
    int soff[EPT];
#pragma unroll
    for (int x = 0; x < EPT; ++x) {
        const int f = tid + 512 * x;
        const int ks = f / (NT * 64), t = (f / 64) % NT, ln = f & 63;
        const int n = n0 + t * 32 + (ln & 31);
        sval[x] = f < NE && n < N;
        srow[x] = Bt + (int64_t)(sval[x] ? n : 0) * B;
        soff[x] = 16 * ks + 8 * (ln >> 5);
    }
    bf16x8_t ones;
#pragma unroll
    for (int j = 0; j < 8; ++j) ones[j] = (__bf16)1.0f;
    f32x16_t acc[NT + 1];
#pragma unroll
    for (int t = 0; t <= NT; ++t) acc[t] = f32x16_t{};

    bf16x8_t stage[EPT], a_next[KS];
    auto fetch = [&](int64_t k0) {
#pragma unroll
        for (int x = 0; x < EPT; ++x) stage[x] = load_frag<VEC>(srow[x], k0 + soff[x], ke, sval[x]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) a_next[ks] = load_frag<VEC>(arow, k0 + 16 * ks + 8 * half, ke, mvalid);
    };
    auto publish = [&](int buf) {
#pragma unroll
        for (int x = 0; x < EPT; ++x)
            if (tid + 512 * x < NE) lds_b[buf][tid + 512 * x] = stage[x];
    };
    fetch(kb);
    publish(0);
    __syncthreads();
    int buf = 0;
    for (int64_t k0 = kb; k0 < ke; k0 += 16 * KS) {
        bf16x8_t a_cur[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) a_cur[ks] = a_next[ks];
        const bool more = k0 + 16 * KS < ke;
        if (more) fetch(k0 + 16 * KS);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (k0 + 16 * ks >= ke) break;
#pragma unroll
            for (int t = 0; t < NT; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_cur[ks], lds_b[buf][(ks * NT + t) * 64 + lane],
                                                                 acc[t], 0, 0, 0);
            if (with_bias) acc[NT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_cur[ks], ones, acc[NT], 0, 0, 0);
        }
        if (more) publish(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }
    const int64_t ld = N + 1;
    float* __restrict__ out = part + (int64_t)s * M * ld;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int mm = mt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (mm >= M) continue;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int nn = n0 + t * 32 + row;
            if (nn < N) out[(int64_t)mm * ld + nn] = acc[t][r];
        }
        if (with_bias && row == 0) out[(int64_t)mm * ld + N] = acc[NT][r];
    }
}

// A single m-tile (the head layer): one wave, no sharing, fragments straight
// from memory.
template <int NT, bool VEC, typename TA = float, typename TB = float>
__global__ __launch_bounds__(64) void wgrad_direct_kernel(const TA* __restrict__ A, const TB* __restrict__ Bt,
                                                         float* __restrict__ part, int M, int N, int32_t B,
                                                         int64_t chunk) {
    const int lane = threadIdx.x & 63, mt = 0;
    const int row = lane & 31, half = lane >> 5;
    const int s = blockIdx.x;
    const int64_t kb = (int64_t)s * chunk;
    const int64_t ke = min(kb + chunk, (int64_t)B);
    const int m = mt * 32 + row;
    const bool mvalid = m < M;
    const TA* __restrict__ arow = A + (int64_t)(mvalid ? m : 0) * B;
    const TB* __restrict__ brow[NT];
    bool nvalid[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int n = t * 32 + row;
        nvalid[t] = n < N;
        brow[t] = Bt + (int64_t)(nvalid[t] ? n : 0) * B;
    }
    bf16x8_t ones;
#pragma unroll
    for (int j = 0; j < 8; ++j) ones[j] = (__bf16)1.0f;
    f32x16_t acc[NT + 1];
#pragma unroll
    for (int t = 0; t <= NT; ++t) acc[t] = f32x16_t{};
    for (int64_t k0 = kb; k0 < ke; k0 += 16) {
        const int64_t k = k0 + 8 * half;
        const bf16x8_t a = load_frag<VEC>(arow, k, ke, mvalid);
        bf16x8_t bb[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) bb[t] = load_frag<VEC>(brow[t], k, ke, nvalid[t]);
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb[t], acc[t], 0, 0, 0);
        acc[NT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ones, acc[NT], 0, 0, 0);
    }
    // accumulator register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
    const int64_t ld = N + 1;
    float* __restrict__ out = part + (int64_t)s * M * ld;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int mm = mt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (mm >= M) continue;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int nn = t * 32 + row;
            if (nn < N) out[(int64_t)mm * ld + nn] = acc[t][r];
        }
        if (row == 0) out[(int64_t)mm * ld + N] = acc[NT][r];
    }
}

// The head's few outputs over many partials: one wave per output; lane l adds
// partials l, l + 64, ... in ascending order, then a fixed shuffle tree.
constexpr int64_t kReduceWaveMax = 4096;          // outputs below which a wave takes each

__global__ __launch_bounds__(256) void wgrad_reduce_wave_kernel(const float* __restrict__ part, int S, int M, int N,
                                                                float* __restrict__ gw, float* __restrict__ gb) {
    const int64_t ld = N + 1, MN = (int64_t)M * ld;
    const int64_t e = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (e >= MN) return;                          // uniform over the wave
    float acc = 0.0f;
    for (int s = lane; s < S; s += 64) acc += part[(int64_t)s * MN + e];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane != 0) return;
    const int64_t mm = e / ld, nn = e - mm * ld;
    if (nn < N) gw[mm * N + nn] = acc;
    else gb[mm] = acc;
}

// grad_w[m][n] (n < N) and grad_b[m] from the partials, summed over s ascending
__global__ void wgrad_reduce_kernel(const float* __restrict__ part, int S, int M, int N, float* __restrict__ gw,
                                    float* __restrict__ gb) {
    const int64_t ld = N + 1, MN = (int64_t)M * ld;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= MN) return;
    float acc = 0.0f;
    int s = 0;
    for (; s + 8 <= S; s += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = part[(int64_t)(s + j) * MN + e];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc += v[j];
    }
    for (; s < S; ++s) acc += part[(int64_t)s * MN + e];
    const int64_t mm = e / ld, nn = e - mm * ld;
    if (nn < N) gw[mm * N + nn] = acc;
    else gb[mm] = acc;
}

// NT n-tiles per workgroup, ny workgroups across N (matrix-core path only).
template <int NT, typename TA, typename TB>
static void launch_wgrad_nt(const TA* A, const TB* Bt, float* part, int M, int N, int32_t B, int S,
                            int64_t chunk, int ny, hipStream_t s) {
    // 16-byte rows: 4 fp32 or 8 bf16 values
    const bool vec = B % (std::is_same<TA, float>::value && std::is_same<TB, float>::value ? 4 : 8) == 0;
    if (M <= 32) {
        if (vec)
            hipLaunchKernelGGL((wgrad_direct_kernel<NT, true, TA, TB>), dim3(S), dim3(64), 0, s, A, Bt, part, M, N, B,
                               chunk);
        else
            hipLaunchKernelGGL((wgrad_direct_kernel<NT, false, TA, TB>), dim3(S), dim3(64), 0, s, A, Bt, part, M, N, B,
                               chunk);
    } else {
        const dim3 grid((uint32_t)S, (uint32_t)ny);
        if (vec)
            hipLaunchKernelGGL((wgrad_mfma_kernel<NT, true, TA, TB>), grid, dim3(512), 0, s, A, Bt, part, M, N, B,
                               chunk);
        else
            hipLaunchKernelGGL((wgrad_mfma_kernel<NT, false, TA, TB>), grid, dim3(512), 0, s, A, Bt, part, M, N, B,
                               chunk);
    }
}

// The gradient of a one-output layer (the head): dW[n] = sum over b of
// g[b] Bt[n][b] and db = sum of g[b], a workgroup per n (the last one the
// bias).  Thread t adds samples 8 t .. 8 t + 7, then 8 t + 8192 .., in
// ascending order, then a fixed tree over the workgroup: the order depends on B
// alone and is the same for bf16 storage and fp32 rows.  The products of bf16
// numbers are exact in fp32, so only the sums round.  VEC (B a multiple of 8,
// rows 16-byte aligned): each thread's eight samples as 16-byte loads.
constexpr int kRowThreads = 1024;

template <bool VEC, typename TB>
__global__ __launch_bounds__(kRowThreads) void wgrad_row_kernel(const float* __restrict__ g,
                                                                const TB* __restrict__ Bt, int N, int32_t B,
                                                                float* __restrict__ gw, float* __restrict__ gb) {
    __shared__ float red[kRowThreads];
    const int n = (int)blockIdx.x;
    const bool bias = n == N;
    const TB* __restrict__ row = Bt + (int64_t)(bias ? 0 : n) * B;
    const int tid = (int)threadIdx.x;
    float acc = 0.0f;
    for (int64_t b0 = (int64_t)tid * 8; b0 < B; b0 += (int64_t)kRowThreads * 8) {
        float gv[8], xv[8];
        if (VEC) {
            const float4 p = *reinterpret_cast<const float4*>(g + b0);
            const float4 q = *reinterpret_cast<const float4*>(g + b0 + 4);
            gv[0] = p.x; gv[1] = p.y; gv[2] = p.z; gv[3] = p.w; gv[4] = q.x; gv[5] = q.y; gv[6] = q.z; gv[7] = q.w;
            if (bias) {
#pragma unroll
                for (int e = 0; e < 8; ++e) xv[e] = 1.0f;
            } else if constexpr (std::is_same<TB, bf16s_t>::value) {
                const uint4 r = *reinterpret_cast<const uint4*>(row + b0);
                const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) xv[e] = __uint_as_float(((w[e >> 1] >> (16 * (e & 1))) & 0xFFFFu) << 16);
            } else {
                const float4 r0 = *reinterpret_cast<const float4*>(row + b0);
                const float4 r1 = *reinterpret_cast<const float4*>(row + b0 + 4);
                xv[0] = r0.x; xv[1] = r0.y; xv[2] = r0.z; xv[3] = r0.w;
                xv[4] = r1.x; xv[5] = r1.y; xv[6] = r1.z; xv[7] = r1.w;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const bool in = b0 + e < B;
                gv[e] = in ? g[b0 + e] : 0.0f;
                xv[e] = in && !bias ? ld_act(row, b0 + e) : 1.0f;
            }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc += gv[e] * xv[e];
    }
    red[tid] = acc;
    __syncthreads();
#pragma unroll
    for (int w = kRowThreads / 2; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    if (tid == 0) {
        if (bias) gb[0] = red[0];
        else gw[n] = red[0];
    }
}

// dW = A Bt^T and db = A 1 for A [M x B], Bt [N x B]; M, N <= 256.  With
// fewer sample chunks than CUs the n-tiles are split over two workgroups per
// chunk (each reads the chunk's A rows, half of its Bt rows).
template <typename TA, typename TB>
static hipError_t weight_grad_mfma(const TA* A, const TB* Bt, int M, int N, int32_t B, float* part,
                                   float* gw, float* gb, int n_cu, hipStream_t s) {
    if constexpr (std::is_same<TA, float>::value) {
        if (M == 1) {                                 // the head: a dot product per weight
            const bool vec = B % 8 == 0 && (reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(Bt)) % 16 == 0;
            if (vec)
                hipLaunchKernelGGL((wgrad_row_kernel<true, TB>), dim3((uint32_t)N + 1), dim3(kRowThreads), 0, s, A, Bt,
                                   N, B, gw, gb);
            else
                hipLaunchKernelGGL((wgrad_row_kernel<false, TB>), dim3((uint32_t)N + 1), dim3(kRowThreads), 0, s, A,
                                   Bt, N, B, gw, gb);
            return hipGetLastError();
        }
    }
    const WgradPlan p = wgrad_plan(B, M);
    const int tiles = (N + 31) / 32;
    const int ny = (M > 32 && tiles >= 2 && p.S < n_cu) ? 2 : 1;
    switch ((tiles + ny - 1) / ny) {
        case 1: launch_wgrad_nt<1>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 2: launch_wgrad_nt<2>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 3: launch_wgrad_nt<3>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 4: launch_wgrad_nt<4>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 5: launch_wgrad_nt<5>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 6: launch_wgrad_nt<6>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 7: launch_wgrad_nt<7>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        case 8: launch_wgrad_nt<8>(A, Bt, part, M, N, B, p.S, p.chunk, ny, s); break;
        default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t MN = (int64_t)M * (N + 1);
    if (MN < kReduceWaveMax)
        hipLaunchKernelGGL(wgrad_reduce_wave_kernel, dim3(blocks_for(MN, 4)), dim3(256), 0, s, part, p.S, M, N, gw, gb);
    else
        hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks_for(MN, 256)), dim3(256), 0, s, part, p.S, M, N, gw, gb);
    return hipGetLastError();
}

// out[e] = sum over s ascending of part[s][e]
__global__ void splitk_reduce_kernel(const float* __restrict__ part, int S, int64_t MN, float* __restrict__ out) {
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= MN) return;
    float acc = 0.0f;
    for (int s = 0; s < S; ++s) acc += part[(int64_t)s * MN + e];
    out[e] = acc;
}

// out[m] = sum_b X[m][b], fixed-order tree per row
__global__ __launch_bounds__(256) void rowsum_kernel(const float* __restrict__ X, int32_t B, float* __restrict__ out) {
    __shared__ float red[256];
    const float* __restrict__ row = X + (int64_t)blockIdx.x * B;
    float s = 0.0f;
    for (int64_t b = threadIdx.x; b < B; b += 256) s += row[b];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[blockIdx.x] = red[0];
}

// D1[m][n] = (Z1[m][n] > 0) ? q(sum_j W[m][j] * D2[j][n]) : 0   (W [M x K], D2 [K x B])
template <bool BF>
__global__ __launch_bounds__(256) void backprop_hidden_kernel(const float* __restrict__ W, const float* __restrict__ D2,
                                                              const uint64_t* __restrict__ Z1, float* __restrict__ D1,
                                                              int M, int K, int32_t B, DropArgs D, int layer) {
    __shared__ float As[16][64 + 4];
    __shared__ float Bs[16][64 + 4];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.y * 64;
    const int64_t n0 = (int64_t)blockIdx.x * 64;
    float acc[4][4] = {};
    const int lrow = tid >> 2, lcol = (tid & 3) * 4;
    const int brow = tid >> 4, bcol = (tid & 15) * 4;
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int kk = k0 + lcol + e, m = m0 + lrow;
            As[lcol + e][lrow] = (m < M && kk < K) ? W[(int64_t)m * K + kk] : 0.0f;
            int kr = k0 + brow;
            int64_t n = n0 + bcol + e;
            Bs[brow][bcol + e] = (kr < K && n < B) ? D2[(int64_t)kr * B + n] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int m = m0 + ty * 4 + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int64_t n = n0 + tx * 4 + j;
            if (n >= B) continue;
            int64_t e = (int64_t)m * B + n;
            const float v = apply_drop(D, layer, n, m, mask_bit(Z1, B, m, n) ? acc[i][j] : 0.0f);
            D1[e] = BF ? q_bf16(v) : v;
        }
    }
}

__global__ void sgd_kernel(float* __restrict__ master, const float* __restrict__ grad, float lr, int64_t n,
                           float* __restrict__ grad_out) {
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    float gr = grad[t];
    master[t] = (float)((double)master[t] - (double)lr * (double)gr);
    if (grad_out) grad_out[t] = gr;
}

static hipError_t weight_grad(const float* A, const float* Bt, int M, int N, int32_t B, const UpdWs& w, float* out,
                              hipStream_t s) {
    dim3 grid((M + 63) / 64, (N + 63) / 64, w.S);
    hipLaunchKernelGGL(gemm_nt_splitk_kernel, grid, dim3(256), 0, s, A, Bt, w.part, M, N, B, w.chunk);
    int64_t MN = (int64_t)M * N;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks_for(MN, 256)), dim3(256), 0, s, w.part, w.S, MN, out);
    return hipGetLastError();
}

// Forward pass of B raw rows in the kernel's precision (the canonical chains),
// keeping every layer feature-major: xn [d][B], a[l] [h_l][B], t [B], and,
// where zb[l] is not null, layer l's ReLU mask.
template <bool BF>
static void forward_rows(const ModelDims& m, const float* compute, const float* mu, const float* isig, int32_t B,
                         const float* feats, float* xn, uint64_t* const* zb, float* const* a, float* t,
                         const DropArgs& D, hipStream_t s) {
    const int64_t nB = B;
    hipLaunchKernelGGL(normalize_kernel<BF>, dim3(blocks_for(nB, 64), (m.d + 63) / 64), dim3(256), 0, s, feats, mu, isig,
                       xn, B, m.d);
    const uint32_t sb = blocks_for(nB, 256);
    const uint32_t sbd = blocks_for(nB, 256 * kDenseSpl);
    bool lds_w = m.d <= kDenseMaxK;
    for (int l = 0; l < m.L; ++l) lds_w = lds_w && m.h[l] <= kDenseMaxK;
    for (int l = 0; l < m.L; ++l) {
        const float* in = l == 0 ? xn : a[l - 1];
        const int K = m.in_of(l), O = m.h[l];
        const int tiles = lds_w ? dense_mfma(m, B, O) : 0;
        if (tiles) {
            launch_dense_mfma<BF, kFwdRelu, float>(tiles, in, compute + m.c_wt[l], compute + m.c_bl[l], zb[l], nullptr, a[l],
                                            B, K, O, D, l, s);
        } else if (lds_w && dense_small(B, O)) {
            if (zb[l]) (void)launch_fill_u64(zb[l], 0ull, (int64_t)O * mask_words(B), s);   // bits set by atomics
            hipLaunchKernelGGL((dense_small_kernel<BF, kFwdRelu>), dim3((O + 63) / 64, blocks_for(nB, 4)), dim3(256), 0,
                               s, in, compute + m.c_wt[l], compute + m.c_bl[l], zb[l], nullptr, a[l], B, K, O, D, l);
        } else if (lds_w) {
            hipLaunchKernelGGL((dense_lane_kernel<BF, kFwdRelu>), dim3(sbd, (O + kDenseUnits - 1) / kDenseUnits),
                               dim3(256), 0, s, in,
                               compute + m.c_wt[l], compute + m.c_bl[l], zb[l], nullptr, a[l], B, K, O, D, l);
        } else {
            hipLaunchKernelGGL((layer_fwd_kernel<BF, true>), dim3(sb, (O + 31) / 32), dim3(256), 0, s, in,
                               compute + m.c_wt[l], compute + m.c_bl[l], nullptr, zb[l], a[l], B, K, O, D, l);
        }
    }
    const float* last = a[m.L - 1];
    if (lds_w && dense_small(B, 1))
        hipLaunchKernelGGL((dense_small_kernel<BF, kFwdHead>), dim3(1, blocks_for(nB, 256)), dim3(256), 0, s, last,
                           compute + m.c_wt[m.L], compute + m.c_bl[m.L], nullptr, t, nullptr, B, m.hl, 1, D, m.L);
    else if (lds_w)
        hipLaunchKernelGGL((dense_lane_kernel<BF, kFwdHead>), dim3(sbd, 1), dim3(256), 0, s, last,
                           compute + m.c_wt[m.L], compute + m.c_bl[m.L], nullptr, t, nullptr, B, m.hl, 1, D, m.L);
    else
        hipLaunchKernelGGL((layer_fwd_kernel<BF, false>), dim3(sb, 1), dim3(256), 0, s, last, compute + m.c_wt[m.L],
                           compute + m.c_bl[m.L], t, nullptr, nullptr, B, m.hl, 1, D, m.L);
}

int64_t forward_rows_floats(const ModelDims& m, int32_t B) {
    int64_t n = (int64_t)B * (m.d + 1) + 64 * (m.L + 2);
    for (int l = 0; l < m.L; ++l) n += (int64_t)B * m.h[l];
    return n;
}

// Carves xn, a[l] and t out of ws (forward_rows_floats floats); scoring keeps no masks.
static float* carve_rows(const ModelDims& m, int32_t B, float* ws, float** xn, float** a) {
    auto take = [&](int64_t n) { float* p = ws; ws += (n + 63) & ~int64_t(63); return p; };
    *xn = take((int64_t)m.d * B);
    for (int l = 0; l < m.L; ++l) a[l] = take((int64_t)m.h[l] * B);
    return take(B);
}

hipError_t launch_forward_rows(const ModelDims& m, const float* compute, const float* mu, const float* isig, int32_t B,
                               const float* feats, float* ws, float** alast_out, float** t_out, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    float *xn, *a[3] = {};
    uint64_t* zb[3] = {};
    float* t = carve_rows(m, B, ws, &xn, a);
    const DropArgs none{};
    if (m.bf16) forward_rows<true>(m, compute, mu, isig, B, feats, xn, zb, a, t, none, s);
    else forward_rows<false>(m, compute, mu, isig, B, feats, xn, zb, a, t, none, s);
    *alast_out = a[m.L - 1];
    *t_out = t;
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// scores of every pair for models other than two hidden layers
// ---------------------------------------------------------------------------
// The pairs' raw feature rows [instance columns | L, n, l, kappa, u], a chunk
// at a time, through the same canonical forward (bias first, inputs in
// ascending order); the two-layer models have fused scorers of their own.
constexpr int64_t kGenericChunk = 1 << 16;

__global__ void pair_rows_kernel(int64_t p0, int64_t P, int32_t N, int d, int d_inst, int block_tokens,
                                 const int64_t* __restrict__ req_off, const int32_t* __restrict__ prompt_len,
                                 const int32_t* __restrict__ overlap, const float* __restrict__ inst_feat,
                                 float* __restrict__ rows) {
    const int64_t total = P * d;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int64_t q = t / d;
        const int c = (int)(t - q * d);
        const int64_t p = p0 + q;
        const int64_t r = p / N;
        const int32_t i = (int32_t)(p - r * N);
        float v;
        if (c < d_inst) {
            v = inst_feat[(int64_t)i * d_inst + c];
        } else {
            float x[5];
            derived_columns(prompt_len[r], req_off[r + 1] - req_off[r], overlap[p], block_tokens, x);
            v = x[c - d_inst];
        }
        rows[t] = v;
    }
}

int64_t generic_score_floats(const ModelDims& m, int64_t pairs) {
    const int32_t P = (int32_t)(pairs < kGenericChunk ? (pairs > 0 ? pairs : 1) : kGenericChunk);
    return (int64_t)P * m.d + forward_rows_floats(m, P) + 64;
}

hipError_t launch_score_generic(const ModelDims& m, const float* compute, const float* mu, const float* isig,
                                int32_t R, int32_t N, const int64_t* req_off, const int32_t* prompt_len,
                                const int32_t* overlap, const float* inst_feat, float* scores, float* ws, int n_cu,
                                hipStream_t s) {
    const int64_t pairs = (int64_t)R * N;
    const DropArgs none{};
    for (int64_t p0 = 0; p0 < pairs; p0 += kGenericChunk) {
        const int32_t P = (int32_t)(pairs - p0 < kGenericChunk ? pairs - p0 : kGenericChunk);
        float* rows = ws;
        float* fw = ws + (((int64_t)P * m.d + 63) & ~int64_t(63));
        int64_t g = ((int64_t)P * m.d + 255) / 256;
        if (g > (int64_t)n_cu * 16) g = (int64_t)n_cu * 16;
        hipLaunchKernelGGL(pair_rows_kernel, dim3((uint32_t)g), dim3(256), 0, s, p0, (int64_t)P, N, m.d, m.d_inst,
                           m.block_tokens, req_off, prompt_len, overlap, inst_feat, rows);
        float *xn, *a[3] = {};
        uint64_t* zb[3] = {};
        (void)carve_rows(m, P, fw, &xn, a);
        if (m.bf16) forward_rows<true>(m, compute, mu, isig, P, rows, xn, zb, a, scores + p0, none, s);
        else forward_rows<false>(m, compute, mu, isig, P, rows, xn, zb, a, scores + p0, none, s);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// the step
// ---------------------------------------------------------------------------
// bf16 models whose hidden layers all run on the matrix-core chains (and B a
// multiple of 8, for 16-byte fragment loads): the same step, with the saved
// normalised inputs, activations and layer gradients stored as bf16 bits.
static hipError_t run_update_b16(const ModelDims& m, float* master, float* compute, const float* mu, const float* isig,
                                 int32_t B, const float* feats, const float* ttft, float lr, float* loss_out,
                                 float* grad_out, const UpdWs& w, const DropArgs& D, int n_cu, hipStream_t s) {
    const int64_t nB = B;
    const int L = m.L;
    bf16s_t* xn = reinterpret_cast<bf16s_t*>(w.xn);
    bf16s_t *a[3] = {}, *dl[3] = {};
    for (int l = 0; l < L; ++l) {
        a[l] = reinterpret_cast<bf16s_t*>(w.a[l]);
        dl[l] = reinterpret_cast<bf16s_t*>(w.dl[l]);
    }
    hipLaunchKernelGGL(normalize_b16_kernel, dim3(blocks_for(nB, 64), (m.d + 63) / 64), dim3(256), 0, s, feats, mu,
                       isig, xn, B, m.d);
    for (int l = 0; l < L; ++l)
        launch_dense_mfma<true, kFwdRelu, bf16s_t>(dense_mfma(m, B, m.h[l]), l == 0 ? xn : a[l - 1],
                                                   compute + m.c_wt[l], compute + m.c_bl[l], w.zb[l], nullptr, a[l], B,
                                                   m.in_of(l), m.h[l], D, l, s);
    hipLaunchKernelGGL((dense_small_kernel<true, kFwdHead, bf16s_t>), dim3(1, blocks_for(nB, 256)), dim3(256), 0, s,
                       a[L - 1], compute + m.c_wt[L], compute + m.c_bl[L], nullptr, w.t, nullptr, B, m.hl, 1, D, L);
    hipLaunchKernelGGL(loss_grad_kernel<true>, dim3(w.loss_blocks), dim3(256), 0, s, w.t, ttft, w.g, w.loss_part, B);
    if (loss_out)
        hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(256), 0, s, w.loss_part, w.loss_blocks, B, loss_out);
    hipError_t e = weight_grad_mfma(w.g, (const bf16s_t*)a[L - 1], 1, m.hl, B, w.part, w.grad + m.m_w[L],
                                    w.grad + m.m_b[L], n_cu, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(delta_head_b16_kernel, dim3(blocks_for(nB, 2048), (m.hl + kDeltaUnits - 1) / kDeltaUnits),
                       dim3(256), 0, s, w.g, compute + m.c_wt[L], w.zb[L - 1], dl[L - 1], B, m.hl, D, L - 1);
    for (int l = L - 1; l >= 0; --l) {
        e = weight_grad_mfma((const bf16s_t*)dl[l], (const bf16s_t*)(l == 0 ? xn : a[l - 1]), m.h[l], m.in_of(l), B,
                             w.part, w.grad + m.m_w[l], w.grad + m.m_b[l], n_cu, s);
        if (e != hipSuccess) return e;
        if (l == 0) break;
        launch_dense_mfma<true, kBackprop, bf16s_t>(dense_mfma(m, B, m.h[l - 1]), dl[l], compute + m.c_wt[l], nullptr,
                                                    w.zb[l - 1], dl[l - 1], nullptr, B, m.h[l], m.h[l - 1], D, l - 1,
                                                    s);
    }
    hipLaunchKernelGGL(sgd_kernel, dim3(blocks_for(m.n_params, 256)), dim3(256), 0, s, master, w.grad, lr,
                       m.n_params, grad_out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_refresh_compute_copy(m, master, compute, s);
}

template <bool BF>
static hipError_t run_update(const ModelDims& m, float* master, float* compute, const float* mu, const float* isig,
                             int32_t B, const float* feats, const float* ttft, float lr, float* loss_out,
                             float* grad_out, void* workspace, const DropArgs& D, int n_cu, hipStream_t s) {
    UpdWs w = plan_ws(m, B, reinterpret_cast<char*>(workspace));
    const int64_t nB = B;
    const int L = m.L;
    bool lds_w = m.d <= kDenseMaxK;
    bool mf = BF && m.d <= 256;          // bf16 operands: weight and bias gradients on the matrix cores
    for (int l = 0; l < L; ++l) {
        lds_w = lds_w && m.h[l] <= kDenseMaxK;
        mf = mf && m.h[l] <= 256;
    }
    bool b16 = BF && mf && lds_w && B % 8 == 0 && dense_small(B, 1);
    for (int l = 0; l < L; ++l) b16 = b16 && dense_mfma(m, B, m.h[l]) > 0;
    if (b16) return run_update_b16(m, master, compute, mu, isig, B, feats, ttft, lr, loss_out, grad_out, w, D, n_cu, s);
    // forward, saving pre-activations and activations (dropout applied)
    forward_rows<BF>(m, compute, mu, isig, B, feats, w.xn, w.zb, w.a, w.t, D, s);
    const uint32_t sbd = blocks_for(nB, 256 * kDenseSpl);
    // loss and output gradient
    hipLaunchKernelGGL(loss_grad_kernel<BF>, dim3(w.loss_blocks), dim3(256), 0, s, w.t, ttft, w.g, w.loss_part, B);
    if (loss_out)
        hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(256), 0, s, w.loss_part, w.loss_blocks, B, loss_out);
    hipError_t e;
    // head
    if (mf) {
        e = weight_grad_mfma(w.g, w.a[L - 1], 1, m.hl, B, w.part, w.grad + m.m_w[L], w.grad + m.m_b[L], n_cu, s);
    } else {
        e = weight_grad(w.g, w.a[L - 1], 1, m.hl, B, w, w.grad + m.m_w[L], s);
        hipLaunchKernelGGL(rowsum_kernel, dim3(1), dim3(256), 0, s, w.g, B, w.grad + m.m_b[L]);
    }
    if (e != hipSuccess) return e;
    if (B % 4 == 0)
        hipLaunchKernelGGL((delta_head_kernel<BF, true>), dim3(blocks_for(nB, 1024), m.hl), dim3(256), 0, s, w.g,
                           compute + m.c_wt[L], w.zb[L - 1], w.dl[L - 1], B, D, L - 1);
    else
        hipLaunchKernelGGL((delta_head_kernel<BF, false>), dim3(blocks_for(nB, 256), m.hl), dim3(256), 0, s, w.g,
                           compute + m.c_wt[L], w.zb[L - 1], w.dl[L - 1], B, D, L - 1);
    // hidden layers, last to first
    for (int l = L - 1; l >= 0; --l) {
        const float* in = l == 0 ? w.xn : w.a[l - 1];
        const int K = m.in_of(l), O = m.h[l];
        if (mf) {
            e = weight_grad_mfma(w.dl[l], in, O, K, B, w.part, w.grad + m.m_w[l], w.grad + m.m_b[l], n_cu, s);
        } else {
            e = weight_grad(w.dl[l], in, O, K, B, w, w.grad + m.m_w[l], s);
            hipLaunchKernelGGL(rowsum_kernel, dim3(O), dim3(256), 0, s, w.dl[l], B, w.grad + m.m_b[l]);
        }
        if (e != hipSuccess) return e;
        if (l == 0) break;
        // dL/dz of layer l - 1 = (W_l^T dL/dz_l), masked by z_{l-1} > 0 and dropout
        const int Kp = m.h[l - 1];
        const int tiles = lds_w ? dense_mfma(m, B, Kp) : 0;
        if (tiles)
            launch_dense_mfma<BF, kBackprop, float>(tiles, w.dl[l], compute + m.c_wt[l], nullptr, w.zb[l - 1], w.dl[l - 1],
                                             nullptr, B, O, Kp, D, l - 1, s);
        else if (lds_w && dense_small(B, Kp))
            hipLaunchKernelGGL((dense_small_kernel<BF, kBackprop>), dim3((Kp + 63) / 64, blocks_for(nB, 4)), dim3(256),
                               0, s, w.dl[l], compute + m.c_wt[l], nullptr, w.zb[l - 1], w.dl[l - 1], nullptr, B, O, Kp,
                               D, l - 1);
        else if (lds_w)
            hipLaunchKernelGGL((dense_lane_kernel<BF, kBackprop>), dim3(sbd, (Kp + kDenseUnits - 1) / kDenseUnits),
                               dim3(256), 0, s, w.dl[l],
                               compute + m.c_wt[l], nullptr, w.zb[l - 1], w.dl[l - 1], nullptr, B, O, Kp, D, l - 1);
        else
            hipLaunchKernelGGL(backprop_hidden_kernel<BF>, dim3(blocks_for(nB, 64), (Kp + 63) / 64), dim3(256), 0, s,
                               compute + m.c_wt[l], w.dl[l], w.zb[l - 1], w.dl[l - 1], Kp, O, B, D, l - 1);
    }
    // step and refresh the compute copy
    hipLaunchKernelGGL(sgd_kernel, dim3(blocks_for(m.n_params, 256)), dim3(256), 0, s, master, w.grad, lr,
                       m.n_params, grad_out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_refresh_compute_copy(m, master, compute, s);
}

hipError_t launch_update(const ModelDims& m, float* master, float* compute, const float* mu,
                         const float* inv_sigma, int32_t B, const float* feats, const float* ttft, float lr,
                         float* loss_out, float* grad_out, void* workspace, const DropArgs& drop, int n_cu,
                         hipStream_t s) {
    if (m.bf16)
        return run_update<true>(m, master, compute, mu, inv_sigma, B, feats, ttft, lr, loss_out, grad_out, workspace,
                                drop, n_cu, s);
    return run_update<false>(m, master, compute, mu, inv_sigma, B, feats, ttft, lr, loss_out, grad_out, workspace,
                             drop, n_cu, s);
}

}  // namespace ls
