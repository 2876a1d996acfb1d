// Online-learning data path (Section 4.3.2, Training-data selection): a FIFO
// of the newest samples and a replay pool that admits the samples the FIFO
// evicts by a gradient-coreset rule, and the gathers of a retraining round.
//
// A sample's embedding is its prediction residual times its last-hidden-layer
// activations, e = (t - y) a_L: the gradient of the squared loss with respect
// to the output weights, up to the factor 2, from the canonical forward of the
// current model (residual in fp32, products and distances in double, each
// distance summed over units in ascending order by one thread).  A candidate
// joins a pool with room; a full pool takes it in place of its most redundant
// member -- the smallest nearest-neighbour distance, lowest slot on ties --
// when the candidate's distance to the pool is larger.  Candidates are decided
// one at a time in eviction order by a single workgroup, since each decision
// depends on the previous ones; the distance work inside a decision is spread
// over the workgroup.
#include "ls_internal.h"

namespace ls {

// Row k of the output comes from A (row code) when code >= 0, else from B
// (row -code - 1).
__global__ void gather_rows_kernel(const int32_t* __restrict__ code, int32_t n, int d, const float* __restrict__ ax,
                                   const float* __restrict__ ay, const float* __restrict__ bx,
                                   const float* __restrict__ by, float* __restrict__ ox, float* __restrict__ oy) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (int64_t)n * (d + 1)) return;
    const int64_t k = e / (d + 1);
    const int c = (int)(e - k * (d + 1));
    const int32_t src = code[k];
    const bool fa = src >= 0;
    const int64_t row = fa ? src : -(int64_t)src - 1;
    if (c < d) ox[k * d + c] = fa ? ax[row * d + c] : bx[row * d + c];
    else oy[k] = fa ? ay[row] : by[row];
}

// Row b of x goes to slot dst[b] of the FIFO when dst[b] >= 0.
__global__ void scatter_rows_kernel(const int32_t* __restrict__ dst, int32_t n, int d, const float* __restrict__ x,
                                    const float* __restrict__ y, float* __restrict__ fx, float* __restrict__ fy) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (int64_t)n * (d + 1)) return;
    const int64_t b = e / (d + 1);
    const int c = (int)(e - b * (d + 1));
    const int32_t slot = dst[b];
    if (slot < 0) return;
    if (c < d) fx[(int64_t)slot * d + c] = x[b * d + c];
    else fy[slot] = y[b];
}

// Embedding of row k (a2 is feature-major [H][n]); rows below n_pool go to the
// pool's table, the rest to the candidates' table.
__global__ void embed_kernel(const float* __restrict__ a2, const float* __restrict__ t, const float* __restrict__ y,
                             int32_t n, int32_t n_pool, int H, double* __restrict__ pool_emb,
                             double* __restrict__ cand_emb) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (int64_t)n * H) return;
    const int64_t k = e / H;
    const int j = (int)(e - k * H);
    const float res = t[k] - y[k];
    const double v = (double)res * (double)a2[(int64_t)j * n + k];
    if (k < n_pool) pool_emb[k * H + j] = v;
    else cand_emb[(k - n_pool) * H + j] = v;
}

__device__ __forceinline__ double emb_dist(const double* __restrict__ a, const double* __restrict__ b, int H) {
    double s = 0.0;
    for (int j = 0; j < H; ++j) {
        const double e = a[j] - b[j];
        s += e * e;
    }
    return s;
}

// Workgroup-wide lexicographic minimum of (value, index); index -1 = none.
constexpr int kAdmitThreads = 1024;

__device__ __forceinline__ void better_pair(double& v, int32_t& i, double ov, int32_t oi) {
    if (oi >= 0 && (i < 0 || ov < v || (ov == v && oi < i))) { v = ov; i = oi; }
}

__device__ void block_min_pair(double& v, int32_t& i, double* sv, int32_t* si) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) better_pair(v, i, __shfl_xor(v, off), __shfl_xor(i, off));
    __syncthreads();
    if (lane == 0) { sv[wv] = v; si[wv] = i; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < (int)(blockDim.x >> 6); ++k) better_pair(sv[0], si[0], sv[k], si[k]);
    }
    __syncthreads();
    v = sv[0];
    i = si[0];
}

// The pool keeps its pairwise distances D [cap x cap] (D[k][k] = +inf), so a
// nearest neighbour is a row minimum.  Every entry is one emb_dist, summed by
// one thread in ascending unit order.
__global__ __launch_bounds__(256) void pool_dist_kernel(const double* __restrict__ emb, int H, int32_t n, int32_t cap,
                                                        double* __restrict__ D) {
    const int32_t i = blockIdx.y;
    const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    D[(int64_t)i * cap + j] = (i == j) ? INFINITY : emb_dist(emb + (int64_t)i * H, emb + (int64_t)j * H, H);
}

// minimum of row k of D over columns [0, n) other than k (lowest column on ties)
__device__ void row_min_block(const double* __restrict__ D, int32_t cap, int32_t n, int32_t k, double* sv, int32_t* si,
                              double* out_d, int32_t* out_i) {
    double v = INFINITY;
    int32_t idx = -1;
    for (int32_t j = threadIdx.x; j < n; j += blockDim.x) {
        if (j == k) continue;
        better_pair(v, idx, D[(int64_t)k * cap + j], j);
    }
    block_min_pair(v, idx, sv, si);
    if (threadIdx.x == 0) {
        *out_d = idx >= 0 ? v : INFINITY;
        *out_i = idx;
    }
    __syncthreads();
}

__global__ __launch_bounds__(256) void pool_nn_kernel(const double* __restrict__ D, int32_t cap, int32_t n,
                                                      double* __restrict__ nnd, int32_t* __restrict__ nni) {
    __shared__ double sv[4];
    __shared__ int32_t si[4];
    row_min_block(D, cap, n, (int32_t)blockIdx.x, sv, si, nnd + blockIdx.x, nni + blockIdx.x);
}

// distances of one candidate to the n current members
__global__ __launch_bounds__(256) void cand_row_kernel(const double* __restrict__ e, const double* __restrict__ emb,
                                                       int H, int32_t n, double* __restrict__ row) {
    const int32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n) row[k] = emb_dist(e, emb + (int64_t)k * H, H);
}

// One decision on a pool of n members (cap slots).  The host knows n: the pool
// grows by one per candidate until it is full and keeps its size afterwards.
__global__ __launch_bounds__(kAdmitThreads) void admit_one_kernel(const double* __restrict__ e,
                                                                  const float* __restrict__ cxr,
                                                                  const float* __restrict__ cyr, int d, int H,
                                                                  int32_t n, int32_t cap,
                                                                  const double* __restrict__ row,
                                                                  double* __restrict__ emb, float* __restrict__ rx,
                                                                  float* __restrict__ ry, double* __restrict__ D,
                                                                  double* __restrict__ nnd, int32_t* __restrict__ nni,
                                                                  int32_t* __restrict__ redo,
                                                                  int32_t* __restrict__ admitted) {
    __shared__ double sv[kAdmitThreads / 64];
    __shared__ int32_t si[kAdmitThreads / 64];
    __shared__ int32_t n_redo;
    int32_t slot, m;
    if (n < cap) {
        slot = n;
        m = n + 1;
    } else {
        double dc = INFINITY, mv = INFINITY;
        int32_t dci = -1, mi = -1;
        for (int32_t k = threadIdx.x; k < n; k += blockDim.x) {
            better_pair(dc, dci, row[k], k);
            better_pair(mv, mi, nnd[k], k);
        }
        block_min_pair(dc, dci, sv, si);
        block_min_pair(mv, mi, sv, si);
        if (!(dc > mv)) return;                             // uniform across the workgroup
        slot = mi;
        m = n;
    }
    for (int j = threadIdx.x; j < H; j += blockDim.x) emb[(int64_t)slot * H + j] = e[j];
    for (int q = threadIdx.x; q < d; q += blockDim.x) rx[(int64_t)slot * d + q] = cxr[q];
    for (int32_t k = threadIdx.x; k < m; k += blockDim.x) {
        const double v = (k == slot) ? INFINITY : row[k];
        D[(int64_t)slot * cap + k] = v;
        D[(int64_t)k * cap + slot] = v;
    }
    if (threadIdx.x == 0) {
        ry[slot] = *cyr;
        n_redo = 0;
        *admitted += 1;
    }
    __syncthreads();
    for (int32_t k = threadIdx.x; k < m; k += blockDim.x) {
        if (k == slot) continue;
        if (nni[k] == slot) {
            redo[atomicAdd(&n_redo, 1)] = k;
        } else {
            const double v = row[k];
            if (v < nnd[k] || (v == nnd[k] && slot < nni[k])) {
                nnd[k] = v;
                nni[k] = slot;
            }
        }
    }
    __syncthreads();
    const int32_t nr = n_redo;
    for (int32_t q = 0; q < nr; ++q) {
        const int32_t k = redo[q];
        row_min_block(D, cap, m, k, sv, si, nnd + k, nni + k);
    }
    row_min_block(D, cap, m, slot, sv, si, nnd + slot, nni + slot);
}

static inline uint32_t grid_of(int64_t n, int block) { return (uint32_t)((n + block - 1) / block); }

hipError_t launch_gather_rows(const int32_t* code, int32_t n, int d, const float* ax, const float* ay,
                              const float* bx, const float* by, float* ox, float* oy, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_of((int64_t)n * (d + 1), 256)), dim3(256), 0, s, code, n, d, ax,
                       ay, bx, by, ox, oy);
    return hipGetLastError();
}

hipError_t launch_scatter_rows(const int32_t* dst, int32_t n, int d, const float* x, const float* y, float* fx,
                               float* fy, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(scatter_rows_kernel, dim3(grid_of((int64_t)n * (d + 1), 256)), dim3(256), 0, s, dst, n, d, x, y,
                       fx, fy);
    return hipGetLastError();
}

hipError_t launch_admission(const float* a2, const float* t, const float* y_all, int32_t n0, int32_t nc, int H, int d,
                            int32_t cap, const float* cx, const float* cy, double* cemb, double* emb, float* rx,
                            float* ry, double* D, double* nnd, int32_t* nni, double* row, int32_t* redo,
                            int32_t* admitted, hipStream_t s) {
    const int32_t n = n0 + nc;
    if (n <= 0 || cap <= 0) return hipSuccess;
    hipLaunchKernelGGL(embed_kernel, dim3(grid_of((int64_t)n * H, 256)), dim3(256), 0, s, a2, t, y_all, n, n0, H, emb,
                       cemb);
    if (n0 > 0) {
        hipLaunchKernelGGL(pool_dist_kernel, dim3(grid_of(n0, 256), (uint32_t)n0), dim3(256), 0, s, emb, H, n0, cap, D);
        hipLaunchKernelGGL(pool_nn_kernel, dim3((uint32_t)n0), dim3(256), 0, s, D, cap, n0, nnd, nni);
    }
    hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(admitted), 0u, 1, s);
    if (e != hipSuccess) return e;
    int32_t size = n0;
    for (int32_t c = 0; c < nc; ++c) {
        if (size > 0)
            hipLaunchKernelGGL(cand_row_kernel, dim3(grid_of(size, 256)), dim3(256), 0, s, cemb + (int64_t)c * H, emb,
                               H, size, row);
        hipLaunchKernelGGL(admit_one_kernel, dim3(1), dim3(kAdmitThreads), 0, s, cemb + (int64_t)c * H,
                           cx + (int64_t)c * d, cy + c, d, H, size, cap, row, emb, rx, ry, D, nnd, nni, redo,
                           admitted);
        if (size < cap) ++size;
    }
    return hipGetLastError();
}

// Mean minibatch loss of a round's last epoch: a running double sum.
__global__ void loss_accumulate_kernel(const float* __restrict__ loss, double* __restrict__ acc, int reset) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *acc = (reset ? 0.0 : *acc) + (double)*loss;
}

__global__ void loss_finish_kernel(const double* __restrict__ acc, int32_t count, float* __restrict__ out) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *out = (float)(*acc / (double)count);
}

hipError_t launch_loss_accumulate(const float* loss, double* acc, int reset, hipStream_t s) {
    hipLaunchKernelGGL(loss_accumulate_kernel, dim3(1), dim3(64), 0, s, loss, acc, reset);
    return hipGetLastError();
}

hipError_t launch_loss_finish(const double* acc, int32_t count, float* out, hipStream_t s) {
    hipLaunchKernelGGL(loss_finish_kernel, dim3(1), dim3(64), 0, s, acc, count, out);
    return hipGetLastError();
}

}  // namespace ls
