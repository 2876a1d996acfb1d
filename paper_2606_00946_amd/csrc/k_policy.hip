// Routing policy around the reward model: the gateway's routing with fallback
// (Alg. 3) and the routing service's logic (Alg. 4), with the heuristic the
// gateway falls back to (Alg. 1, prefix-cache-and-load, or Alg. 2, prefix-aware
// with a threshold).  One wave decides one request from its row of overlaps
// and scores; the per-instance request counts, their mean and standard
// deviation and the cluster's KV saturation are shared by every request and
// computed once per batch, in ascending instance order, so every rounding is
// the same as in a sequential evaluation.
#include "k_policy.h"

namespace ls {

__device__ __forceinline__ bool in_bounds(float v, float lo, float hi) { return lo <= v && v <= hi; }

// One workgroup: request counts, out-of-range instances, batch statistics.
__global__ __launch_bounds__(256) void policy_stats_kernel(PolicyArgs P, const float* __restrict__ inst_feat, int32_t N,
                                                           int d_inst, double* __restrict__ cnt,
                                                           PolicyStats* __restrict__ st) {
    __shared__ int any_ood;
    if (threadIdx.x == 0) any_ood = 0;
    __syncthreads();
    for (int32_t i = threadIdx.x; i < N; i += blockDim.x) {
        const float* row = inst_feat + (int64_t)i * d_inst;
        double ci = 0.0;
        if (P.count_col0 >= 0) ci += (double)row[P.count_col0];
        if (P.count_col1 >= 0) ci += (double)row[P.count_col1];
        cnt[i] = ci;
        if (P.lo) {
            bool ok = true;
            for (int c = 0; c < d_inst; ++c) ok &= in_bounds(row[c], P.lo[c], P.hi[c]);
            if (!ok) atomicOr(&any_ood, 1);
        }
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    double cmin = cnt[0], cmax = cnt[0], sum = 0.0, kv = 0.0;
    for (int32_t i = 0; i < N; ++i) {
        const double c = cnt[i];
        if (c < cmin) cmin = c;
        if (c > cmax) cmax = c;
        sum += c;
        if (P.kv_col >= 0) kv += (double)inst_feat[(int64_t)i * d_inst + P.kv_col];
    }
    const double mu = sum / (double)N;
    double var = 0.0;
    for (int32_t i = 0; i < N; ++i) {
        const double e = cnt[i] - mu;
        var += e * e;
    }
    const double sigma = sqrt(var / (double)N);
    PolicyStats s;
    s.limit = mu + P.overload_k * sigma;
    s.imbalanced = (cmax - cmin > P.theta_imbal) ? 1 : 0;
    s.saturated = (P.kv_col >= 0 && kv / (double)N > P.tau_sat) ? 1 : 0;
    s.any_inst_ood = any_ood;
    *st = s;
}

// (value, id) reductions across a wave; ids >= N mark empty lanes.
__device__ __forceinline__ void wave_min_count(double& c, int32_t& id) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const double oc = __shfl_xor(c, off);
        const int32_t oi = __shfl_xor(id, off);
        if (oc < c || (oc == c && oi < id)) { c = oc; id = oi; }
    }
}

// best prefix match: larger m, then smaller c, then lower id
__device__ __forceinline__ void wave_best_match(float& m, double& c, int32_t& id) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float om = __shfl_xor(m, off);
        const double oc = __shfl_xor(c, off);
        const int32_t oi = __shfl_xor(id, off);
        const bool take = oi != INT_MAX &&
                          (id == INT_MAX || om > m || (om == m && (oc < c || (oc == c && oi < id))));
        if (take) { m = om; c = oc; id = oi; }
    }
}

__device__ __forceinline__ void wave_argmin_score(float& t, int32_t& id) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float ot = __shfl_xor(t, off);
        const int32_t oi = __shfl_xor(id, off);
        if (better(ot, oi, t, id)) { t = ot; id = oi; }
    }
}

__device__ __forceinline__ float hit_ratio(int32_t L, int32_t l, int block_tokens) {
    const int64_t hit = (int64_t)block_tokens * l;
    return (L == 0) ? 0.0f : (float)hit / (float)L;
}

__global__ __launch_bounds__(256) void route_kernel(PolicyArgs P, const PolicyStats* __restrict__ stp,
                                                    const double* __restrict__ cnt, int32_t R, int32_t N, int d_inst,
                                                    int block_tokens, const int64_t* __restrict__ req_off,
                                                    const uint64_t* __restrict__ req_hashes,
                                                    const int32_t* __restrict__ prompt_len,
                                                    const int32_t* __restrict__ overlap,
                                                    const float* __restrict__ scores, const uint8_t* __restrict__ band,
                                                    const float* __restrict__ inst_feat,
                                                    const uint32_t* __restrict__ rnd, int32_t* __restrict__ chosen,
                                                    int32_t* __restrict__ status, int32_t* __restrict__ heur_out,
                                                    float* __restrict__ feat_out) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (r >= R) return;
    const PolicyStats st = *stp;
    const int32_t L = prompt_len[r];
    const int64_t n = req_off[r + 1] - req_off[r];
    const int32_t* __restrict__ ov = overlap + r * N;
    const float* __restrict__ sc = scores + r * N;
    const uint8_t* __restrict__ bd = band ? band + r * N : nullptr;

    // ---- the heuristic (Alg. 1 or Alg. 2) and the request's best prefix benefit
    double lc = INFINITY;               // least loaded
    int32_t li = INT_MAX;
    float bm = 0.0f;                    // best match (Alg. 1: among the not overloaded; Alg. 2: overall)
    double bc = 0.0;
    int32_t bi = INT_MAX;
    double kl = -INFINITY;              // max_i kappa_i * L
    for (int32_t i = lane; i < N; i += 64) {
        const double c = cnt[i];
        const float m = hit_ratio(L, ov[i], block_tokens);
        kl = fmax(kl, (double)m * (double)L);
        if (c < lc || (c == lc && i < li)) { lc = c; li = i; }
        const bool eligible = P.heuristic == 2 || c <= st.limit;
        if (eligible && (bi == INT_MAX || m > bm || (m == bm && (P.heuristic == 2 ? false : c < bc)))) {
            bm = m; bc = c; bi = i;
        }
    }
    wave_min_count(lc, li);
    if (P.heuristic == 2) bc = 0.0;     // Alg. 2 orders by match, then id only
    wave_best_match(bm, bc, bi);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) kl = fmax(kl, __shfl_xor(kl, off));
    int32_t heur;
    if (P.heuristic == 2) heur = ((double)bm > P.prefix_tau) ? bi : li;
    else if (st.imbalanced) heur = li;
    else heur = bi != INT_MAX ? bi : li;

    // ---- Alg. 3 / Alg. 4
    int32_t pick, code;
    bool ood = false;
    if (P.lo) {
        ood = !in_bounds((float)L, P.lo[d_inst], P.hi[d_inst]) || !in_bounds((float)n, P.lo[d_inst + 1], P.hi[d_inst + 1]) ||
              st.any_inst_ood;
    }
    const uint32_t* __restrict__ u = rnd ? rnd + 3 * r : nullptr;
    if (P.cold) {
        pick = heur; code = LS_ROUTE_COLD_START;
    } else if (ood) {
        pick = heur; code = LS_ROUTE_OOD;
    } else if (u && (uint64_t)u[0] < P.explore_thr) {
        pick = (int32_t)(((uint64_t)u[1] * (uint64_t)N) >> 32);
        code = LS_ROUTE_OK | LS_ROUTE_EXPLORED;
    } else {
        code = LS_ROUTE_OK;
        // greedy: argmin of the (canonical) candidate scores
        float bt = 0.0f;
        int32_t bid = INT_MAX;
        for (int32_t i = lane; i < N; i += 64) {
            if (bd && !bd[i]) continue;
            if (better(sc[i], i, bt, bid)) { bt = sc[i]; bid = i; }
        }
        wave_argmin_score(bt, bid);
        // K-filter
        int32_t C[LS_MAX_KFILTER];
        int nc = 0;
        if (P.k_filter > 0 && n >= 1 && st.saturated && kl > P.tau_ben) {
            nc = hrw_topk_wave(req_hashes[req_off[r]], N, P.k_filter, C, lane);
            code |= LS_ROUTE_KFILTER;
            bool inC = false;
            for (int q = 0; q < nc; ++q) inC |= (C[q] == bid);
            if (!inC) {
                int32_t b2 = C[0];
                for (int q = 1; q < nc; ++q)
                    if (better(sc[C[q]], C[q], sc[b2], b2)) b2 = C[q];
                bid = b2;
            }
            bt = sc[bid];
        }
        pick = bid;
        // near-best tie-break
        if (P.delta >= 0.0 && !(bt != bt)) {
            const double lim = (double)bt + P.delta * fabs((double)bt);
            uint32_t total = 0;
            for (int32_t i0 = 0; i0 < N; i0 += 64) {
                const int32_t i = i0 + lane;
                bool mem = false;
                if (i < N && (!bd || bd[i])) {
                    bool scope = nc == 0;
                    for (int q = 0; q < nc; ++q) scope |= (C[q] == i);
                    mem = scope && (double)sc[i] <= lim;
                }
                total += (uint32_t)__popcll(__ballot(mem));
            }
            if (total > 1) {
                uint32_t k = (uint32_t)(((uint64_t)u[2] * (uint64_t)total) >> 32);
                for (int32_t i0 = 0; i0 < N; i0 += 64) {
                    const int32_t i = i0 + lane;
                    bool mem = false;
                    if (i < N && (!bd || bd[i])) {
                        bool scope = nc == 0;
                        for (int q = 0; q < nc; ++q) scope |= (C[q] == i);
                        mem = scope && (double)sc[i] <= lim;
                    }
                    const uint64_t m = __ballot(mem);
                    const uint32_t cm = (uint32_t)__popcll(m);
                    if (k < cm) {
                        uint64_t mm = m;
                        for (uint32_t t = 0; t < k; ++t) mm &= mm - 1;      // drop the k lowest members
                        pick = i0 + __ffsll((long long)mm) - 1;
                        break;
                    }
                    k -= cm;
                }
                code |= LS_ROUTE_TIEBREAK;
            }
        }
    }
    if (lane == 0) {
        chosen[r] = pick;
        if (status) status[r] = code;
        if (heur_out) heur_out[r] = heur;
    }
    if (feat_out) {
        const int d = d_inst + 5;
        float* dst = feat_out + r * d;
        for (int c = lane; c < d_inst; c += 64) dst[c] = inst_feat[(int64_t)pick * d_inst + c];
        if (lane == 0) {
            float x[5];
            derived_columns(L, n, ov[pick], block_tokens, x);
            for (int c = 0; c < 5; ++c) dst[d_inst + c] = x[c];
        }
    }
}

hipError_t launch_policy_stats(const PolicyArgs& P, const float* inst_feat, int32_t N, int d_inst, double* cnt,
                               PolicyStats* st, hipStream_t s) {
    hipLaunchKernelGGL(policy_stats_kernel, dim3(1), dim3(256), 0, s, P, inst_feat, N, d_inst, cnt, st);
    return hipGetLastError();
}

hipError_t launch_route(const PolicyArgs& P, const PolicyStats* st, const double* cnt, const ModelDims& m, int32_t R,
                        int32_t N, const int64_t* req_off, const uint64_t* req_hashes, const int32_t* prompt_len,
                        const int32_t* overlap, const float* scores, const uint8_t* band, const float* inst_feat,
                        const uint32_t* rnd, int32_t* chosen, int32_t* status, int32_t* heur, float* feat_out,
                        hipStream_t s) {
    if (R <= 0) return hipSuccess;
    hipLaunchKernelGGL(route_kernel, dim3((uint32_t)(((int64_t)R + 3) / 4)), dim3(256), 0, s, P, st, cnt, R, N, m.d_inst,
                       m.block_tokens, req_off, req_hashes, prompt_len, overlap, scores, band, inst_feat, rnd, chosen,
                       status, heur, feat_out);
    return hipGetLastError();
}

}  // namespace ls
