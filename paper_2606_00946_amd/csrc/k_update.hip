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

#include "ls_internal.h"

namespace ls {

__device__ __forceinline__ float q_bf16(float x) {
    if (x != x) return x;
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

__device__ __forceinline__ float relu_u(float z) { return z > 0.0f ? z : 0.0f; }

static inline uint32_t blocks_for(int64_t n, int block) { return (uint32_t)((n + block - 1) / block); }

// ---------------------------------------------------------------------------
// workspace layout
// ---------------------------------------------------------------------------
struct UpdWs {
    float *xn, *z1, *a1, *z2, *a2, *t, *g, *d2, *d1, *grad, *part, *loss_part;
    int64_t bytes;
    int S;              // split-K chunks
    int64_t chunk;      // samples per chunk (multiple of 16)
    int loss_blocks;
};

static int64_t align_floats(int64_t n) { return (n + 63) & ~int64_t(63); }

static UpdWs plan_ws(const ModelDims& m, int32_t B, char* base) {
    UpdWs w{};
    int S = B / 1024;
    if (S < 1) S = 1;
    if (S > 128) S = 128;
    int64_t chunk = ((int64_t)B + S - 1) / S;
    chunk = (chunk + 15) & ~int64_t(15);
    S = (int)(((int64_t)B + chunk - 1) / chunk);
    w.S = S;
    w.chunk = chunk;
    w.loss_blocks = (int)blocks_for(B, 256);
    int64_t maxmn = std::max<int64_t>({(int64_t)m.h2 * m.h1, (int64_t)m.h1 * m.d, (int64_t)m.h2});
    int64_t sizes[] = {(int64_t)m.d * B, (int64_t)m.h1 * B, (int64_t)m.h1 * B, (int64_t)m.h2 * B,
                       (int64_t)m.h2 * B, (int64_t)B, (int64_t)B, (int64_t)m.h2 * B, (int64_t)m.h1 * B,
                       m.n_params, (int64_t)S * maxmn, (int64_t)w.loss_blocks};
    float** slots[] = {&w.xn, &w.z1, &w.a1, &w.z2, &w.a2, &w.t, &w.g, &w.d2, &w.d1, &w.grad, &w.part, &w.loss_part};
    int64_t off = 0;
    for (int k = 0; k < 12; ++k) {
        *slots[k] = base ? reinterpret_cast<float*>(base) + off : nullptr;
        off += align_floats(sizes[k]);
    }
    w.bytes = off * (int64_t)sizeof(float);
    return w;
}

int64_t update_workspace_bytes(const ModelDims& m, int32_t B) { return plan_ws(m, B, nullptr).bytes; }

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <bool BF>
__global__ void normalize_kernel(const float* __restrict__ feats, const float* __restrict__ mu,
                                 const float* __restrict__ isig, float* __restrict__ xn, int32_t B, int d) {
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)B * d) return;
    int64_t c = t / B, b = t - c * B;
    float v = __fmul_rn(__fsub_rn(feats[b * d + c], mu[c]), isig[c]);
    xn[t] = BF ? q_bf16(v) : v;
}

template <bool BF, bool RELU, int U>
__device__ __forceinline__ void fwd_units(const float* __restrict__ in, const float* __restrict__ wt,
                                          const float* __restrict__ bias, float* __restrict__ z,
                                          float* __restrict__ a, int32_t B, int K, int O, int jb, int64_t b,
                                          bool valid) {
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = bias[jb + u];
    for (int k = 0; k < K; ++k) {
        float x = in[(int64_t)k * B + b];
        const float* __restrict__ w = wt + (int64_t)k * O + jb;
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] = __builtin_fmaf(w[u], x, acc[u]);
    }
    if (!valid) return;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        z[(int64_t)(jb + u) * B + b] = acc[u];
        if (RELU) {
            float h = relu_u(acc[u]);
            a[(int64_t)(jb + u) * B + b] = BF ? q_bf16(h) : h;
        }
    }
}

// One layer for every sample: lane = sample, weights uniform across the wave.
template <bool BF, bool RELU>
__global__ __launch_bounds__(256) void layer_fwd_kernel(const float* __restrict__ in, const float* __restrict__ wt,
                                                        const float* __restrict__ bias, float* __restrict__ z,
                                                        float* __restrict__ a, int32_t B, int K, int O) {
    int64_t bt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool valid = bt < B;
    int64_t b = valid ? bt : 0;
    int jb = 0;
    for (; jb + 32 <= O; jb += 32) fwd_units<BF, RELU, 32>(in, wt, bias, z, a, B, K, O, jb, b, valid);
    if (jb + 16 <= O) { fwd_units<BF, RELU, 16>(in, wt, bias, z, a, B, K, O, jb, b, valid); jb += 16; }
    if (jb + 8 <= O) { fwd_units<BF, RELU, 8>(in, wt, bias, z, a, B, K, O, jb, b, valid); jb += 8; }
    if (jb + 4 <= O) { fwd_units<BF, RELU, 4>(in, wt, bias, z, a, B, K, O, jb, b, valid); jb += 4; }
    if (jb + 2 <= O) { fwd_units<BF, RELU, 2>(in, wt, bias, z, a, B, K, O, jb, b, valid); jb += 2; }
    if (jb + 1 <= O) { fwd_units<BF, RELU, 1>(in, wt, bias, z, a, B, K, O, jb, b, valid); jb += 1; }
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

// dL/dz of the last hidden layer: g_b * w3[j] where z2 > 0
template <bool BF>
__global__ void delta_head_kernel(const float* __restrict__ g, const float* __restrict__ w3,
                                  const float* __restrict__ z2, float* __restrict__ d2, int32_t B, int h2) {
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)h2 * B) return;
    int64_t j = t / B, b = t - j * B;
    float v = z2[t] > 0.0f ? g[b] * w3[j] : 0.0f;
    d2[t] = BF ? q_bf16(v) : v;
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
                                                              const float* __restrict__ Z1, float* __restrict__ D1,
                                                              int M, int K, int32_t B) {
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
            float v = Z1[e] > 0.0f ? acc[i][j] : 0.0f;
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

template <bool BF>
static hipError_t run_update(const ModelDims& m, float* master, float* compute, const float* mu, const float* isig,
                             int32_t B, const float* feats, const float* ttft, float lr, float* loss_out,
                             float* grad_out, void* workspace, hipStream_t s) {
    UpdWs w = plan_ws(m, B, reinterpret_cast<char*>(workspace));
    const int64_t nB = B;
    // forward, saving pre-activations and activations
    hipLaunchKernelGGL(normalize_kernel<BF>, dim3(blocks_for(nB * m.d, 256)), dim3(256), 0, s, feats, mu, isig, w.xn,
                       B, m.d);
    hipLaunchKernelGGL((layer_fwd_kernel<BF, true>), dim3(blocks_for(nB, 256)), dim3(256), 0, s, w.xn,
                       compute + m.c_w1t, compute + m.c_b1, w.z1, w.a1, B, m.d, m.h1);
    hipLaunchKernelGGL((layer_fwd_kernel<BF, true>), dim3(blocks_for(nB, 256)), dim3(256), 0, s, w.a1,
                       compute + m.c_w2t, compute + m.c_b2, w.z2, w.a2, B, m.h1, m.h2);
    hipLaunchKernelGGL((layer_fwd_kernel<BF, false>), dim3(blocks_for(nB, 256)), dim3(256), 0, s, w.a2,
                       compute + m.c_w3, compute + m.c_b3, w.t, nullptr, B, m.h2, 1);
    // loss and output gradient
    hipLaunchKernelGGL(loss_grad_kernel<BF>, dim3(w.loss_blocks), dim3(256), 0, s, w.t, ttft, w.g, w.loss_part, B);
    if (loss_out)
        hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(256), 0, s, w.loss_part, w.loss_blocks, B, loss_out);
    // head layer
    hipError_t e = weight_grad(w.g, w.a2, 1, m.h2, B, w, w.grad + m.m_w3, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rowsum_kernel, dim3(1), dim3(256), 0, s, w.g, B, w.grad + m.m_b3);
    // second hidden layer
    hipLaunchKernelGGL(delta_head_kernel<BF>, dim3(blocks_for(nB * m.h2, 256)), dim3(256), 0, s, w.g,
                       compute + m.c_w3, w.z2, w.d2, B, m.h2);
    e = weight_grad(w.d2, w.a1, m.h2, m.h1, B, w, w.grad + m.m_w2, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rowsum_kernel, dim3(m.h2), dim3(256), 0, s, w.d2, B, w.grad + m.m_b2);
    // first hidden layer
    hipLaunchKernelGGL(backprop_hidden_kernel<BF>, dim3(blocks_for(nB, 64), (m.h1 + 63) / 64), dim3(256), 0, s,
                       compute + m.c_w2t, w.d2, w.z1, w.d1, m.h1, m.h2, B);
    e = weight_grad(w.d1, w.xn, m.h1, m.d, B, w, w.grad + m.m_w1, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rowsum_kernel, dim3(m.h1), dim3(256), 0, s, w.d1, B, w.grad + m.m_b1);
    // step and refresh the compute copy
    hipLaunchKernelGGL(sgd_kernel, dim3(blocks_for(m.n_params, 256)), dim3(256), 0, s, master, w.grad, lr,
                       m.n_params, grad_out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_refresh_compute_copy(m, master, compute, s);
}

hipError_t launch_update(const ModelDims& m, float* master, float* compute, const float* mu,
                         const float* inv_sigma, int32_t B, const float* feats, const float* ttft, float lr,
                         float* loss_out, float* grad_out, void* workspace, hipStream_t s) {
    if (m.bf16)
        return run_update<true>(m, master, compute, mu, inv_sigma, B, feats, ttft, lr, loss_out, grad_out, workspace, s);
    return run_update<false>(m, master, compute, mu, inv_sigma, B, feats, ttft, lr, loss_out, grad_out, workspace, s);
}

}  // namespace ls
