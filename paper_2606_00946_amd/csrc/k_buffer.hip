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
// one at a time in eviction order, since each decision depends on the previous
// ones, but the distances they need do not: for a chunk of candidates the
// distances to the pool as it stands and among the chunk are computed up front
// by a tiled kernel over the whole GPU, and one workgroup then walks the chunk,
// taking each distance from the first table or, for a slot a candidate of the
// chunk has taken, from the second.
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

// Workgroup-wide lexicographic minimum of (value, index); index -1 = none.
constexpr int kAdmitThreads = 1024;
constexpr int32_t kAdmitChunk = 256;          // candidates whose distances are computed together
constexpr int kLdsStateCap = 6144;            // largest pool whose per-slot state fits in LDS (144 KB)

__device__ __forceinline__ void better_pair(double& v, int32_t& i, double ov, int32_t oi) {
    if (oi >= 0 && (i < 0 || ov < v || (ov == v && oi < i))) { v = ov; i = oi; }
}

__device__ __forceinline__ void block_min_pair(double& v, int32_t& i, double* sv, int32_t* si) {
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
// nearest neighbour is a row minimum.
//
// out[a * ldo + b] = emb_dist(A_a, B_b) for a < na, b < nb (+inf where a == b
// when `diag`).  A workgroup computes a 16 x 64 tile; rows are staged through
// LDS 32 units at a time and every thread keeps its four sums in registers, so
// each distance is still summed over units in ascending order by one thread.
constexpr int kDistA = 16, kDistB = 64, kDistJ = 32;

__global__ __launch_bounds__(256) void dist_tile_kernel(const double* __restrict__ A, int32_t na,
                                                        const double* __restrict__ B, int32_t nb, int H,
                                                        double* __restrict__ out, int64_t ldo, int diag) {
    __shared__ double sa[kDistA][kDistJ];
    __shared__ double sb[kDistB][kDistJ + 1];
    const int tid = threadIdx.x;
    const int32_t a0 = (int32_t)blockIdx.y * kDistA, b0 = (int32_t)blockIdx.x * kDistB;
    const int bl = tid & 63, ag = tid >> 6;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int j0 = 0; j0 < H; j0 += kDistJ) {
        __syncthreads();
        for (int x = tid; x < kDistA * kDistJ; x += 256) {
            const int r = x / kDistJ, q = x - r * kDistJ;
            const int32_t ar = a0 + r;
            const int j = j0 + q;
            sa[r][q] = (ar < na && j < H) ? A[(int64_t)ar * H + j] : 0.0;
        }
        for (int x = tid; x < kDistB * kDistJ; x += 256) {
            const int r = x / kDistJ, q = x - r * kDistJ;
            const int32_t br = b0 + r;
            const int j = j0 + q;
            sb[r][q] = (br < nb && j < H) ? B[(int64_t)br * H + j] : 0.0;
        }
        __syncthreads();
        const int jn = H - j0 < kDistJ ? H - j0 : kDistJ;
        for (int q = 0; q < jn; ++q) {
            const double bv = sb[bl][q];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const double e = sa[4 * ag + u][q] - bv;
                acc[u] += e * e;
            }
        }
    }
    const int32_t b = b0 + bl;
    if (b >= nb) return;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int32_t ar = a0 + 4 * ag + u;
        if (ar < na) out[(int64_t)ar * ldo + b] = (diag && ar == b) ? INFINITY : acc[u];
    }
}

// minimum of row k of D over columns [0, n) other than k (lowest column on ties)
__device__ __forceinline__ void row_min_block(const double* __restrict__ D, int32_t cap, int32_t n, int32_t k,
                                              double* sv, int32_t* si, double* out_d, int32_t* out_i) {
    double v = INFINITY;
    int32_t idx = -1;
    // eight loads of the row in flight per thread (past the end: a clamped,
    // in-bounds index whose value is ignored)
    constexpr int U = 8;
    for (int32_t j0 = threadIdx.x; j0 < n; j0 += U * blockDim.x) {
        double x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t j = j0 + u * (int32_t)blockDim.x;
            x[u] = D[(int64_t)k * cap + (j < n ? j : n - 1)];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t j = j0 + u * (int32_t)blockDim.x;
            if (j < n && j != k) better_pair(v, idx, x[u], j);
        }
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

// Block-wide lexicographic minima of P (value, index) pairs at once, with two
// barriers for all of them; every thread gets the results.  sv, si: P * 16.
template <int P>
__device__ __forceinline__ void block_min_pairs(double (&v)[P], int32_t (&ix)[P], double* sv, int32_t* si) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int p = 0; p < P; ++p) {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) better_pair(v[p], ix[p], __shfl_xor(v[p], off), __shfl_xor(ix[p], off));
    }
    if (lane == 0) {
#pragma unroll
        for (int p = 0; p < P; ++p) {
            sv[p * 16 + wv] = v[p];
            si[p * 16 + wv] = ix[p];
        }
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < P; ++p) {
        double a = lane < nw ? sv[p * 16 + lane] : INFINITY;
        int32_t b = lane < nw ? si[p * 16 + lane] : -1;
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) better_pair(a, b, __shfl_xor(a, off), __shfl_xor(b, off));
        v[p] = __shfl(a, 0);
        ix[p] = __shfl(b, 0);
    }
    __syncthreads();
}

// One decision, for candidate c of the chunk, on a pool of n members (cap
// slots); row[0 .. n) are the candidate's distances to the members.  The
// workgroup decides together; returns the slot taken, or -1.
//
// D is kept row-major, and an admission writes only its new row: writing the
// column as well would be cap scattered stores in this single workgroup.
// Within a chunk the valid copy of D[k][j] is therefore in the row of
// whichever of k and j was admitted later -- org[] holds the chunk-local
// admission index (-1: not since the chunk started) -- and a multi-workgroup
// pass copies the new rows into their columns after the chunk.
__device__ __forceinline__ int32_t admit_one(int32_t c, const double* __restrict__ e, const float* __restrict__ cxr,
                                             const float* __restrict__ cyr, int d, int H, int32_t n, int32_t cap,
                                             const double* row, double* __restrict__ emb, float* __restrict__ rx,
                                             float* __restrict__ ry, double* __restrict__ D, double* nnd, int32_t* nni,
                                             int32_t* org, int32_t* __restrict__ redo, int32_t* __restrict__ admitted,
                                             int32_t* __restrict__ rslots, int32_t* __restrict__ n_rslots, double* sv,
                                             int32_t* si, int32_t* n_redo) {
    int32_t slot, m;
    if (n < cap) {
        slot = n;
        m = n + 1;
    } else {
        double pv[2] = {INFINITY, INFINITY};
        int32_t pi[2] = {-1, -1};
        for (int32_t k = threadIdx.x; k < n; k += blockDim.x) {
            better_pair(pv[0], pi[0], row[k], k);
            better_pair(pv[1], pi[1], nnd[k], k);
        }
        block_min_pairs<2>(pv, pi, sv, si);
        if (!(pv[0] > pv[1])) return -1;                    // uniform across the workgroup
        slot = pi[1];
        m = n;
    }
    for (int j = threadIdx.x; j < H; j += blockDim.x) emb[(int64_t)slot * H + j] = e[j];
    for (int q = threadIdx.x; q < d; q += blockDim.x) rx[(int64_t)slot * d + q] = cxr[q];
    for (int32_t k = threadIdx.x; k < m; k += blockDim.x) D[(int64_t)slot * cap + k] = (k == slot) ? INFINITY : row[k];
    if (threadIdx.x == 0) {
        ry[slot] = *cyr;
        *n_redo = 0;
        *admitted += 1;
        if (org[slot] < 0) rslots[(*n_rslots)++] = slot;
        org[slot] = c;
    }
    __syncthreads();
    for (int32_t k = threadIdx.x; k < m; k += blockDim.x) {
        if (k == slot) continue;
        if (nni[k] == slot) {
            redo[atomicAdd(n_redo, 1)] = k;
        } else {
            const double v = row[k];
            if (v < nnd[k] || (v == nnd[k] && slot < nni[k])) {
                nnd[k] = v;
                nni[k] = slot;
            }
        }
    }
    __syncthreads();
    // nearest neighbours recomputed for the members that had the replaced one,
    // then for the new member: eight rows per pass over the members
    const int32_t nr = *n_redo;
    constexpr int P = 8;
    for (int32_t q0 = 0; q0 <= nr; q0 += P) {
        int32_t kq[P], ok[P];
        double pv[P];
        int32_t pi[P];
#pragma unroll
        for (int p = 0; p < P; ++p) {
            kq[p] = q0 + p < nr ? redo[q0 + p] : (q0 + p == nr ? slot : -1);
            ok[p] = kq[p] >= 0 ? org[kq[p]] : 0;
            pv[p] = INFINITY;
            pi[p] = -1;
        }
        for (int32_t j = threadIdx.x; j < m; j += blockDim.x) {
            const int32_t oj = org[j];
            double x[P];
#pragma unroll
            for (int p = 0; p < P; ++p) {                // every load in bounds; inactive rows read slot 0
                const int32_t k = kq[p] >= 0 ? kq[p] : 0;
                const bool jrow = oj > ok[p];
                x[p] = kq[p] == slot ? row[j == slot ? 0 : j]
                                     : D[(int64_t)(jrow ? j : k) * cap + (jrow ? k : j)];
            }
#pragma unroll
            for (int p = 0; p < P; ++p)
                if (kq[p] >= 0 && j != kq[p]) better_pair(pv[p], pi[p], x[p], j);
        }
        block_min_pairs<P>(pv, pi, sv, si);
        if (threadIdx.x < P && kq[threadIdx.x] >= 0) {
            const int p = threadIdx.x;
            nnd[kq[p]] = pi[p] >= 0 ? pv[p] : INFINITY;
            nni[kq[p]] = pi[p];
        }
        __syncthreads();
    }
    return slot;
}

// Decides the nch candidates of one chunk in order, on a pool of n members at
// the chunk's start.  dcp[c][k] (row stride cap) is candidate c's distance to
// the member in slot k at the chunk's start, dcc[c][c'] (stride nch) its
// distance to candidate c'.  origin[k] ends as the chunk-local index of the
// last candidate that took slot k (-1: none), rslots / n_rslots as the list of
// slots taken.  With CAPL > 0 (cap <= CAPL) the per-slot state -- nearest-
// neighbour distances and slots, origins, the current candidate's distances --
// lives in LDS for the whole chunk; otherwise in global memory (origin
// cleared by the caller).
template <int CAPL>
__global__ __launch_bounds__(kAdmitThreads) void admit_chunk_kernel(
    const double* __restrict__ cemb, const float* __restrict__ cx, const float* __restrict__ cy, int d, int H,
    int32_t n, int32_t cap, int32_t nch, const double* __restrict__ dcp, const double* __restrict__ dcc,
    int32_t* __restrict__ origin, double* __restrict__ row, double* __restrict__ emb, float* __restrict__ rx,
    float* __restrict__ ry, double* __restrict__ D, double* __restrict__ nnd, int32_t* __restrict__ nni,
    int32_t* __restrict__ redo, int32_t* __restrict__ admitted, int32_t* __restrict__ rslots,
    int32_t* __restrict__ n_rslots) {
    constexpr bool kLds = CAPL > 0;
    constexpr int L = kLds ? CAPL : 1;
    __shared__ double sv[8 * 16];
    __shared__ int32_t si[8 * 16];
    __shared__ int32_t n_redo;
    __shared__ double l_nnd[L], l_row[L];
    __shared__ int32_t l_nni[L], l_org[L];
    double* nnd_w = kLds ? l_nnd : nnd;
    double* row_w = kLds ? l_row : row;
    int32_t* nni_w = kLds ? l_nni : nni;
    int32_t* org_w = kLds ? l_org : origin;
    if (kLds) {
        for (int32_t k = threadIdx.x; k < cap; k += blockDim.x) {
            l_org[k] = -1;
            if (k < n) {
                l_nnd[k] = nnd[k];
                l_nni[k] = nni[k];
            }
        }
    }
    if (threadIdx.x == 0) *n_rslots = 0;
    __syncthreads();
    for (int32_t c = 0; c < nch; ++c) {
        for (int32_t k0 = threadIdx.x; k0 < n; k0 += 8 * blockDim.x) {
            double x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {            // clamped indices keep every load in bounds
                const int32_t k = k0 + u * (int32_t)blockDim.x;
                const int32_t kk = k < n ? k : n - 1;
                const int32_t o = org_w[kk];
                x[u] = o < 0 ? dcp[(int64_t)c * cap + kk] : dcc[(int64_t)c * nch + o];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int32_t k = k0 + u * (int32_t)blockDim.x;
                if (k < n) row_w[k] = x[u];
            }
        }
        __syncthreads();
        (void)admit_one(c, cemb + (int64_t)c * H, cx + (int64_t)c * d, cy + c, d, H, n, cap, row_w, emb, rx, ry, D,
                        nnd_w, nni_w, org_w, redo, admitted, rslots, n_rslots, sv, si, &n_redo);
        if (n < cap) ++n;
        __syncthreads();
    }
    if (kLds) {
        for (int32_t k = threadIdx.x; k < n; k += blockDim.x) {
            nnd[k] = l_nnd[k];
            nni[k] = l_nni[k];
            origin[k] = l_org[k];
        }
    }
}

// After a chunk: every slot the chunk took gets its row copied into its
// column, D[k][s] = D[s][k], except where k was taken later (its own row
// already holds the pair).  Block y handles listed slot y; threads the k.
__global__ __launch_bounds__(256) void flush_columns_kernel(const int32_t* __restrict__ rslots,
                                                            const int32_t* __restrict__ n_rslots,
                                                            const int32_t* __restrict__ origin, int32_t n, int32_t cap,
                                                            double* __restrict__ D) {
    if ((int32_t)blockIdx.y >= *n_rslots) return;
    const int32_t s = rslots[blockIdx.y];
    const int32_t k = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
    if (k >= n || k == s) return;
    if (origin[s] > origin[k]) D[(int64_t)k * cap + s] = D[(int64_t)s * cap + k];
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

int32_t admission_chunk(int32_t nc) { return nc < kAdmitChunk ? nc : kAdmitChunk; }

hipError_t launch_admission(const float* a2, const float* t, const float* y_all, int32_t n0, int32_t nc, int H, int d,
                            int32_t cap, const float* cx, const float* cy, double* cemb, double* emb, float* rx,
                            float* ry, double* D, double* nnd, int32_t* nni, double* row, int32_t* redo,
                            int32_t* admitted, double* dcp, double* dcc, int32_t* origin, int32_t* rslots,
                            hipStream_t s) {
    const int32_t n = n0 + nc;
    if (n <= 0 || cap <= 0) return hipSuccess;
    hipLaunchKernelGGL(embed_kernel, dim3(grid_of((int64_t)n * H, 256)), dim3(256), 0, s, a2, t, y_all, n, n0, H, emb,
                       cemb);
    if (n0 > 0) {
        hipLaunchKernelGGL(dist_tile_kernel, dim3(grid_of(n0, kDistB), grid_of(n0, kDistA)), dim3(256), 0, s, emb, n0,
                           emb, n0, H, D, (int64_t)cap, 1);
        hipLaunchKernelGGL(pool_nn_kernel, dim3((uint32_t)n0), dim3(256), 0, s, D, cap, n0, nnd, nni);
    }
    hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(admitted), 0u, 1, s);
    if (e != hipSuccess) return e;
    const int32_t chunk = admission_chunk(nc);
    int32_t size = n0;
    for (int32_t c0 = 0; c0 < nc; c0 += chunk) {
        const int32_t nch = nc - c0 < chunk ? nc - c0 : chunk;
        const double* ce = cemb + (int64_t)c0 * H;
        if (size > 0)
            hipLaunchKernelGGL(dist_tile_kernel, dim3(grid_of(size, kDistB), grid_of(nch, kDistA)), dim3(256), 0, s, ce,
                               nch, emb, size, H, dcp, (int64_t)cap, 0);
        hipLaunchKernelGGL(dist_tile_kernel, dim3(grid_of(nch, kDistB), grid_of(nch, kDistA)), dim3(256), 0, s, ce, nch,
                           ce, nch, H, dcc, (int64_t)nch, 0);
        if (cap <= kLdsStateCap) {
            hipLaunchKernelGGL(admit_chunk_kernel<kLdsStateCap>, dim3(1), dim3(kAdmitThreads), 0, s, ce,
                               cx + (int64_t)c0 * d, cy + c0, d, H, size, cap, nch, dcp, dcc, origin, row, emb, rx, ry,
                               D, nnd, nni, redo, admitted, rslots, rslots + chunk);
        } else {
            if ((e = launch_fill_u32(reinterpret_cast<uint32_t*>(origin), 0xffffffffu, cap, s)) != hipSuccess) return e;
            hipLaunchKernelGGL(admit_chunk_kernel<0>, dim3(1), dim3(kAdmitThreads), 0, s, ce, cx + (int64_t)c0 * d,
                               cy + c0, d, H, size, cap, nch, dcp, dcc, origin, row, emb, rx, ry, D, nnd, nni, redo,
                               admitted, rslots, rslots + chunk);
        }
        size = size + nch < cap ? size + nch : cap;
        if (c0 + nch < nc)                           // the last chunk's columns are never read
            hipLaunchKernelGGL(flush_columns_kernel, dim3(grid_of(size, 256), (uint32_t)nch), dim3(256), 0, s, rslots,
                               rslots + chunk, origin, size, cap, D);
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
