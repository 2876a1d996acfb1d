// Exact decisions on top of the matrix-core scores: per request, select every
// pair whose fast score could still be the argmin within its error band, and
// rescore those pairs with the canonical fp32 chain (bias first, inputs in
// ascending order), so that the decision and its score are the canonical ones.
//
// The fast scorer writes, for each pair, its score t and an error scale
// E = kBandRel * (sum_j |w3_j| h2_j + |b3|).  A pair is a candidate if
// t - E <= min over the request of (t + E); the argmin then runs over the
// candidates' canonical scores only.
#include "k_policy.h"

namespace ls {

// ---------------------------------------------------------------------------
// band selection and canonical rescoring
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool finite_f(float x) { return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u; }

// One wave per request, 16 requests per workgroup: U = min_i (t_i + E_i) over
// finite pairs; a pair is a candidate if t_i - E_i <= U (or if t_i or E_i is
// not finite).  Candidates are appended to one list with a single atomic per
// workgroup.
constexpr int kBandWaves = 16;

__device__ __forceinline__ bool band_member(float ti, float ei, float U) {
    return !(finite_f(ti) && finite_f(ei)) || (ti - ei <= U);
}

// Policy extensions (routing with the full Alg. 4): with a tie-break margin
// delta >= 0 the bound grows to cover every pair that can be near-best, and
// with the K-filter possible the K instances of the request's prefix group are
// candidates too.
struct BandPolicy {
    double delta;                       // < 0: none
    int32_t k_filter;                   // 0: none
    const PolicyStats* stats;           // saturation flag (K-filter only)
    const int64_t* req_off;
    const uint64_t* req_hashes;
};

// Lane l holds pairs i0 + 4l .. i0 + 4l + 3 of each chunk of 256 (VEC, N a
// multiple of 4: 16-byte reads of t and E, and the four flags written as one
// word), else pairs i0 + l.  The list is in ascending pair order either way.
template <bool VEC>
__global__ __launch_bounds__(1024) void band_select_kernel(int32_t R, int32_t N, const float* __restrict__ t,
                                                           const float* __restrict__ E, BandPolicy BP,
                                                           uint8_t* __restrict__ band, int64_t* __restrict__ list,
                                                           uint32_t* __restrict__ count) {
    constexpr int V = VEC ? 4 : 1;                  // pairs per lane and chunk
    constexpr int CH = 64 * V;                      // chunk
    __shared__ uint32_t wcount[kBandWaves];
    __shared__ uint32_t wbase[kBandWaves];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t r = (int64_t)blockIdx.x * kBandWaves + wv;
    const bool live = r < R;
    const float* __restrict__ tr = t + (live ? r : 0) * N;
    const float* __restrict__ er = E + (live ? r : 0) * N;
    auto load = [&](const float* __restrict__ row, int i, float (&v)[V]) {
        if constexpr (VEC) {
            const float4 q = *reinterpret_cast<const float4*>(row + i);
            v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        } else {
            v[0] = row[i];
        }
    };
    float U = INFINITY, L0 = INFINITY;
    uint32_t cnt = 0;
    int32_t C[LS_MAX_KFILTER];
    int nc = 0;
    if (live) {
        for (int i0 = 0; i0 < N; i0 += CH) {
            const int i = i0 + V * lane;
            if (i < N) {
                float tv[V], ev[V];
                load(tr, i, tv);
                load(er, i, ev);
#pragma unroll
                for (int j = 0; j < V; ++j)
                    if (finite_f(tv[j]) && finite_f(ev[j])) {
                        U = fminf(U, tv[j] + ev[j]);
                        L0 = fminf(L0, tv[j] - ev[j]);
                    }
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            U = fminf(U, __shfl_xor(U, off));
            L0 = fminf(L0, __shfl_xor(L0, off));
        }
        if (BP.delta >= 0.0 && finite_f(U)) {
            // the smallest canonical score lies in [L0, U]; c + delta |c| is largest at an end
            const double a = (double)U + BP.delta * fabs((double)U);
            const double b = (double)L0 + BP.delta * fabs((double)L0);
            U = (float)(a > b ? a : b);
        }
        U = U + fabsf(U) * 0x1p-20f;                // absorbs the rounding of the sums above
        if (BP.k_filter > 0 && BP.stats->saturated && BP.req_off[r + 1] > BP.req_off[r])
            nc = hrw_topk_wave(BP.req_hashes[BP.req_off[r]], N, BP.k_filter, C, lane);
        for (int i0 = 0; i0 < N; i0 += CH) {
            const int i = i0 + V * lane;
            uint32_t bits = 0;
            if (i < N) {
                float tv[V], ev[V];
                load(tr, i, tv);
                load(er, i, ev);
#pragma unroll
                for (int j = 0; j < V; ++j) {
                    bool in = band_member(tv[j], ev[j], U);
                    for (int q = 0; q < nc; ++q) in |= (C[q] == i + j);
                    bits |= (in ? 1u : 0u) << (8 * j);
                }
                if constexpr (VEC) *reinterpret_cast<uint32_t*>(band + r * N + i) = bits;
                else band[r * N + i] = (uint8_t)bits;
            }
            cnt += (uint32_t)__popc(bits);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off);
    }
    if (lane == 0) wcount[wv] = cnt;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t total = 0;
        for (int k = 0; k < kBandWaves; ++k) total += wcount[k];
        uint32_t base = total ? atomicAdd(count, total) : 0u;
        for (int k = 0; k < kBandWaves; ++k) {
            wbase[k] = base;
            base += wcount[k];
        }
    }
    __syncthreads();
    if (!live) return;
    uint32_t base = wbase[wv];
    for (int i0 = 0; i0 < N; i0 += CH) {
        const int i = i0 + V * lane;
        uint32_t bits = 0;
        if (i < N) {
            if constexpr (VEC) bits = *reinterpret_cast<const uint32_t*>(band + r * N + i);
            else bits = band[r * N + i];
        }
        const uint32_t mine = (uint32_t)__popc(bits);
        uint32_t incl = mine;                           // inclusive scan over the lanes
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t up = __shfl_up(incl, d);
            if (lane >= d) incl += up;
        }
        uint32_t pos = base + incl - mine;
#pragma unroll
        for (int j = 0; j < V; ++j)
            if ((bits >> (8 * j)) & 1u) list[pos++] = r * N + i + j;
        base += __shfl(incl, 63);
    }
}

hipError_t launch_band_select(int32_t R, int32_t N, const float* t, const float* E, uint8_t* band, int64_t* list,
                              uint32_t* count, hipStream_t s) {
    return launch_band_select_policy(R, N, t, E, -1.0, 0, nullptr, nullptr, nullptr, band, list, count, s);
}

hipError_t launch_band_select_policy(int32_t R, int32_t N, const float* t, const float* E, double delta,
                                     int32_t k_filter, const PolicyStats* stats, const int64_t* req_off,
                                     const uint64_t* req_hashes, uint8_t* band, int64_t* list, uint32_t* count,
                                     hipStream_t s) {
    if (R <= 0) return hipSuccess;
    BandPolicy BP{delta, k_filter, stats, req_off, req_hashes};
    const dim3 grid((uint32_t)(((int64_t)R + kBandWaves - 1) / kBandWaves)), block(64 * kBandWaves);
    const bool vec = N % 4 == 0 && ((uintptr_t)t | (uintptr_t)E) % 16 == 0 && (uintptr_t)band % 4 == 0;
    if (vec) hipLaunchKernelGGL(band_select_kernel<true>, grid, block, 0, s, R, N, t, E, BP, band, list, count);
    else hipLaunchKernelGGL(band_select_kernel<false>, grid, block, 0, s, R, N, t, E, BP, band, list, count);
    return hipGetLastError();
}

// Two-stage selection for scoring calls.  Stage 1 lists each request's fast
// argmin (smallest finite t, lowest id on ties) for canonical rescoring; its
// canonical score c1 is then an upper bound of the request's canonical minimum.
// Stage 2 keeps every pair whose canonical score can still be <= c1 (or, with a
// tie-break margin delta, within the near-best set's largest bound
// c1 + delta |c1|): t - E <= that bound, a non-finite t or E, or one of the
// K-filter's instances.  With |t - c| <= E for every pair this holds the
// canonical argmin, every exact tie with it and every near-best member, and it
// is about half as wide as the band around min (t + E), which has to allow for
// the best pair's own error as well.
// A wave takes kLeadRows consecutive requests, and every lane's loads for all
// of them go out before any comparison.  VEC (N a multiple of 4, t 16-byte
// aligned): lane l reads pairs i0 + 4l .. i0 + 4l + 3 of each chunk of 256 as
// one 16-byte load.
constexpr int kLeadRows = 4;

template <bool VEC>
__global__ __launch_bounds__(64 * kBandWaves) void band_lead_kernel(int32_t R, int32_t N, const float* __restrict__ t,
                                                                    int64_t* __restrict__ lead) {
    constexpr int V = VEC ? 4 : 1, CH = 64 * V;
    const int lane = threadIdx.x & 63;
    const int64_t r0 = ((int64_t)blockIdx.x * kBandWaves + (threadIdx.x >> 6)) * kLeadRows;
    if (r0 >= R) return;                          // uniform over the wave
    float best[kLeadRows];
    int bi[kLeadRows];                            // N: no finite score seen
#pragma unroll
    for (int k = 0; k < kLeadRows; ++k) {
        best[k] = INFINITY;
        bi[k] = N;
    }
    for (int i0 = 0; i0 < N; i0 += CH) {
        const int i = i0 + V * lane;
        float v[kLeadRows][V];
#pragma unroll
        for (int k = 0; k < kLeadRows; ++k) {
            const bool ok = r0 + k < R && i < N;
            const float* __restrict__ tr = t + (r0 + k) * N;
            if constexpr (VEC) {
                const float4 q = ok ? *reinterpret_cast<const float4*>(tr + i) : float4{INFINITY, INFINITY, INFINITY, INFINITY};
                v[k][0] = q.x; v[k][1] = q.y; v[k][2] = q.z; v[k][3] = q.w;
            } else {
                v[k][0] = ok ? tr[i] : INFINITY;
            }
        }
#pragma unroll
        for (int k = 0; k < kLeadRows; ++k)
#pragma unroll
            for (int j = 0; j < V; ++j) {
                const float x = v[k][j];
                if (i + j < N && finite_f(x) && (x < best[k] || (x == best[k] && i + j < bi[k]))) {
                    best[k] = x;
                    bi[k] = i + j;
                }
            }
    }
#pragma unroll
    for (int k = 0; k < kLeadRows; ++k) {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float ov = __shfl_xor(best[k], off);
            const int oi = __shfl_xor(bi[k], off);
            if (ov < best[k] || (ov == best[k] && oi < bi[k])) {
                best[k] = ov;
                bi[k] = oi;
            }
        }
        if (lane == 0 && r0 + k < R) lead[r0 + k] = (r0 + k) * N + (bi[k] < N ? bi[k] : 0);
    }
}

template <bool VEC>
__global__ __launch_bounds__(1024) void band_rest_kernel(int32_t R, int32_t N, const float* __restrict__ t,
                                                         const float* __restrict__ E, const float* __restrict__ canon,
                                                         const int64_t* __restrict__ lead, BandPolicy BP,
                                                         uint8_t* __restrict__ band, int64_t* __restrict__ list,
                                                         uint32_t* __restrict__ count) {
    constexpr int V = VEC ? 4 : 1;
    constexpr int CH = 64 * V;
    __shared__ uint32_t wcount[kBandWaves];
    __shared__ uint32_t wbase[kBandWaves];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t r = (int64_t)blockIdx.x * kBandWaves + wv;
    const bool live = r < R;
    const float* __restrict__ tr = t + (live ? r : 0) * N;
    const float* __restrict__ er = E + (live ? r : 0) * N;
    auto load = [&](const float* __restrict__ row, int i, float (&v)[V]) {
        if constexpr (VEC) {
            const float4 q = *reinterpret_cast<const float4*>(row + i);
            v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        } else {
            v[0] = row[i];
        }
    };
    int i1 = -1;
    bool all = false;
    float thr = 0.0f;
    int32_t C[LS_MAX_KFILTER];
    int nc = 0;
    uint32_t cnt = 0;
    if (live) {
        const int64_t l1 = lead[r];
        i1 = (int)(l1 - r * N);
        const float c1 = canon[l1];
        if (!finite_f(c1)) {
            // +inf or NaN: any finite canonical score beats it; -inf: only -inf ties
            all = c1 != -INFINITY;
            thr = c1;
        } else if (BP.delta >= 0.0) {
            // c + delta |c| grows with c, so the near-best bound of the true minimum is at most this
            const double b = (double)c1 + BP.delta * fabs((double)c1);
            float f = (float)b;
            if ((double)f < b) f = nextafterf(f, INFINITY);
            thr = f;
        } else {
            thr = c1;     // fl(t - E) <= c1 whenever t - E <= c1: rounding is monotone and c1 is a float
        }
        if (BP.k_filter > 0 && BP.stats->saturated && BP.req_off[r + 1] > BP.req_off[r])
            nc = hrw_topk_wave(BP.req_hashes[BP.req_off[r]], N, BP.k_filter, C, lane);
        for (int i0 = 0; i0 < N; i0 += CH) {
            const int i = i0 + V * lane;
            uint32_t bits = 0, listed = 0;
            if (i < N) {
                float tv[V], ev[V];
                load(tr, i, tv);
                load(er, i, ev);
#pragma unroll
                for (int j = 0; j < V; ++j) {
                    bool in = all || !(finite_f(tv[j]) && finite_f(ev[j])) || (tv[j] - ev[j] <= thr);
                    for (int q = 0; q < nc; ++q) in |= (C[q] == i + j);
                    const bool lead_pair = i + j == i1;
                    bits |= ((in || lead_pair) ? 1u : 0u) << (8 * j);
                    listed |= ((in && !lead_pair) ? 1u : 0u) << (8 * j);
                }
                if constexpr (VEC) *reinterpret_cast<uint32_t*>(band + r * N + i) = bits;
                else band[r * N + i] = (uint8_t)bits;
            }
            cnt += (uint32_t)__popc(listed);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off);
    }
    if (lane == 0) wcount[wv] = cnt;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t total = 0;
        for (int k = 0; k < kBandWaves; ++k) total += wcount[k];
        uint32_t base = total ? atomicAdd(count, total) : 0u;
        for (int k = 0; k < kBandWaves; ++k) {
            wbase[k] = base;
            base += wcount[k];
        }
    }
    __syncthreads();
    if (!live) return;
    uint32_t base = wbase[wv];
    for (int i0 = 0; i0 < N; i0 += CH) {
        const int i = i0 + V * lane;
        uint32_t bits = 0;
        if (i < N) {
            if constexpr (VEC) bits = *reinterpret_cast<const uint32_t*>(band + r * N + i);
            else bits = band[r * N + i];
            if (i1 >= i && i1 < i + V) bits &= ~(1u << (8 * (i1 - i)));     // the lead pair is rescored already
        }
        const uint32_t mine = (uint32_t)__popc(bits);
        uint32_t incl = mine;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t up = __shfl_up(incl, d);
            if (lane >= d) incl += up;
        }
        uint32_t pos = base + incl - mine;
#pragma unroll
        for (int j = 0; j < V; ++j)
            if ((bits >> (8 * j)) & 1u) list[pos++] = r * N + i + j;
        base += __shfl(incl, 63);
    }
}

hipError_t launch_band_lead(int32_t R, int32_t N, const float* t, int64_t* lead, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    const int64_t per = (int64_t)kBandWaves * kLeadRows;
    const dim3 grid((uint32_t)(((int64_t)R + per - 1) / per)), block(64 * kBandWaves);
    if (N % 4 == 0 && (uintptr_t)t % 16 == 0) hipLaunchKernelGGL(band_lead_kernel<true>, grid, block, 0, s, R, N, t, lead);
    else hipLaunchKernelGGL(band_lead_kernel<false>, grid, block, 0, s, R, N, t, lead);
    return hipGetLastError();
}

hipError_t launch_band_rest(int32_t R, int32_t N, const float* t, const float* E, const float* canon,
                            const int64_t* lead, double delta, int32_t k_filter, const PolicyStats* stats,
                            const int64_t* req_off, const uint64_t* req_hashes, uint8_t* band, int64_t* list,
                            uint32_t* count, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    BandPolicy BP{delta, k_filter, stats, req_off, req_hashes};
    const dim3 grid((uint32_t)(((int64_t)R + kBandWaves - 1) / kBandWaves)), block(64 * kBandWaves);
    const bool vec = N % 4 == 0 && ((uintptr_t)t | (uintptr_t)E) % 16 == 0 && (uintptr_t)band % 4 == 0;
    if (vec)
        hipLaunchKernelGGL(band_rest_kernel<true>, grid, block, 0, s, R, N, t, E, canon, lead, BP, band, list, count);
    else
        hipLaunchKernelGGL(band_rest_kernel<false>, grid, block, 0, s, R, N, t, E, canon, lead, BP, band, list, count);
    return hipGetLastError();
}

// Canonical score of every listed pair, written over its fast score.
template <bool BF>
__global__ __launch_bounds__(256) void rescore_kernel(PairModel M, const float* __restrict__ mu,
                                                      const float* __restrict__ isig,
                                                      const float* __restrict__ part_t, int32_t N,
                                                      const int64_t* __restrict__ req_off,
                                                      const int32_t* __restrict__ prompt_len,
                                                      const int32_t* __restrict__ overlap, int block_tokens,
                                                      const int64_t* __restrict__ list,
                                                      const uint32_t* __restrict__ count, float* __restrict__ scores) {
    const uint32_t cnt = *count;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < cnt; q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = list[q];
        const int64_t r = p / N, i = p - r * N;
        float x[5], xt[5];
        derived_columns(prompt_len[r], req_off[r + 1] - req_off[r], overlap[p], block_tokens, x);
        normalise_tail<BF>(x, mu, isig, M.d_inst, xt);
        scores[p] = canonical_score<BF>(M, part_t + i, N, xt);
    }
}

// Same scores, one wave per listed pair (bf16 model, h1 = h2 = H): lanes own
// output units, W2 sits in LDS as bf16 bits, the pair's layer-1 activations
// and then its layer-2 outputs pass through a per-wave LDS row, and lane 0
// runs the head chain.  Every chain keeps the canonical order (bias first,
// inputs ascending), so each score is bitwise the one-lane-per-pair value.
struct RescoreArgs {
    const float* __restrict__ w1;     // [H x d] compute copy
    const float* __restrict__ w2t;    // [H x H] W2T[k][j]
    const float* __restrict__ b2;
    const float* __restrict__ w3;
    const float* __restrict__ b3;
    const float* __restrict__ mu;
    const float* __restrict__ isig;
    const float* __restrict__ part_t;  // [H x N]
    const int64_t* __restrict__ req_off;
    const int32_t* __restrict__ prompt_len;
    const int32_t* __restrict__ overlap;
    const int64_t* __restrict__ list;
    const uint32_t* __restrict__ count;
    float* __restrict__ scores;
    int32_t N;
    int d, d_inst, block_tokens;
};

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Each wave scores four pairs at once, so every weight it converts from bf16
// feeds four chains and the four head chains run side by side.  W2 (as bf16
// bits, 128 KB at H = 256) and eight waves' rows (four pairs x H fp32) fill the
// 160 KB of LDS: two waves per SIMD, so that one wave's layer-1 loads and head
// chains overlap the other's layer-2 FMAs; each block of four inputs' operands
// is read one block ahead of its FMAs.  (Eight pairs per wave at one wave per
// SIMD leaves those serial phases exposed and is slower.)
constexpr int kRescoreWaves = 8;
constexpr int kRescorePairs = 4;

template <int H>
__global__ __launch_bounds__(64 * kRescoreWaves, 1) void rescore_wave_kernel(RescoreArgs A) {
    constexpr int U = H / 64;                  // units per lane
    constexpr int P = kRescorePairs;
    constexpr int RS = H;
    static_assert(U == 1 || U == 2 || U == 4, "H in {64, 128, 256}");
    __shared__ __align__(16) uint16_t lds_w2[H * H];
    __shared__ __align__(16) float lds_row[kRescoreWaves][P][RS];
    {
        // W2 into LDS as bf16 bits: 16-byte loads, eight in flight per thread
        // before any is used (one memory round trip per eight, not per element)
        constexpr int NV = H * H / 4, T = 64 * kRescoreWaves, B8 = 8;
        const float4* __restrict__ src = reinterpret_cast<const float4*>(A.w2t);
        uint2* dst = reinterpret_cast<uint2*>(lds_w2);
        for (int base = threadIdx.x; base < NV; base += T * B8) {
            float4 v[B8];
#pragma unroll
            for (int j = 0; j < B8; ++j)
                if (base + j * T < NV) v[j] = src[base + j * T];
#pragma unroll
            for (int j = 0; j < B8; ++j)
                if (base + j * T < NV)
                    dst[base + j * T] =
                        make_uint2((__float_as_uint(v[j].x) >> 16) | (__float_as_uint(v[j].y) & 0xffff0000u),
                                   (__float_as_uint(v[j].z) >> 16) | (__float_as_uint(v[j].w) & 0xffff0000u));
        }
    }
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    float w1c[U][5], b2v[U];
#pragma unroll
    for (int v = 0; v < U; ++v) {
#pragma unroll
        for (int c = 0; c < 5; ++c) w1c[v][c] = A.w1[(int64_t)(lane + 64 * v) * A.d + A.d_inst + c];
        b2v[v] = A.b2[U * lane + v];
    }
    const float b3 = A.b3[0];
    const int64_t cnt = *A.count;
    float (*rows)[RS] = lds_row[wave];
    for (int64_t q = ((int64_t)blockIdx.x * kRescoreWaves + wave) * P; q < cnt;
         q += (int64_t)gridDim.x * kRescoreWaves * P) {
        int64_t pp[P];
#pragma unroll
        for (int e = 0; e < P; ++e) pp[e] = A.list[q + e < cnt ? q + e : q];
        // layer 1, resumed from the instance partial: unit lane + 64 v
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int64_t r = pp[e] / A.N, i = pp[e] - r * A.N;
            float x[5], xt[5];
            derived_columns(A.prompt_len[r], A.req_off[r + 1] - A.req_off[r], A.overlap[pp[e]], A.block_tokens, x);
            normalise_tail<true>(x, A.mu, A.isig, A.d_inst, xt);
#pragma unroll
            for (int v = 0; v < U; ++v) {
                const int k = lane + 64 * v;
                float z = A.part_t[(int64_t)k * A.N + i];
#pragma unroll
                for (int c = 0; c < 5; ++c) z = __builtin_fmaf(w1c[v][c], xt[c], z);
                rows[e][k] = bf16_rne_num(relu(z));
            }
        }
        wave_sync();
        // layer 2: units U lane .. U lane + U - 1, inputs ascending
        float acc[P][U];
#pragma unroll
        for (int e = 0; e < P; ++e)
#pragma unroll
            for (int u = 0; u < U; ++u) acc[e][u] = b2v[u];
        auto load_block = [&](int k, float4 (&av)[P], uint32_t (&wb)[4][(U + 1) / 2]) {
#pragma unroll
            for (int e = 0; e < P; ++e) av[e] = *reinterpret_cast<const float4*>(&rows[e][k]);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const uint16_t* wr = lds_w2 + (k + kk) * H + U * lane;
                if constexpr (U == 4) {
                    const uint2 w2 = *reinterpret_cast<const uint2*>(wr);
                    wb[kk][0] = w2.x;
                    wb[kk][1] = w2.y;
                } else if constexpr (U == 2) {
                    wb[kk][0] = *reinterpret_cast<const uint32_t*>(wr);
                } else {
                    wb[kk][0] = wr[0];
                }
            }
        };
        auto fma_block = [&](const float4 (&a4)[P], const uint32_t (&wbk)[4][(U + 1) / 2]) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                float wv[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t bits = wbk[kk][u >> 1];
                    wv[u] = __uint_as_float((u & 1) ? (bits & 0xffff0000u) : (bits << 16));
                }
#pragma unroll
                for (int e = 0; e < P; ++e) {
                    const float a = kk == 0 ? a4[e].x : kk == 1 ? a4[e].y : kk == 2 ? a4[e].z : a4[e].w;
#pragma unroll
                    for (int u = 0; u < U; ++u) acc[e][u] = __builtin_fmaf(wv[u], a, acc[e][u]);
                }
            }
        };
        // two operand buffers in turn: block k + 4's reads are issued before block k's FMAs
        float4 av[P], an[P];
        uint32_t wb[4][(U + 1) / 2], wn[4][(U + 1) / 2];
        load_block(0, av, wb);
        for (int k = 0; k < H; k += 8) {
            load_block(k + 4, an, wn);
            fma_block(av, wb);
            if (k + 8 < H) load_block(k + 8, av, wb);
            fma_block(an, wn);
        }
        wave_sync();
#pragma unroll
        for (int e = 0; e < P; ++e) {
            if constexpr (U == 4) {
                *reinterpret_cast<float4*>(&rows[e][4 * lane]) =
                    make_float4(bf16_rne_num(relu(acc[e][0])), bf16_rne_num(relu(acc[e][1])),
                                bf16_rne_num(relu(acc[e][2])), bf16_rne_num(relu(acc[e][3])));
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) rows[e][U * lane + u] = bf16_rne_num(relu(acc[e][u]));
            }
        }
        wave_sync();
        // head: lane e < P runs pair e's chain over the units in ascending order
        if (lane < P && q + lane < cnt) {
            const float* hrow = rows[lane];
            float t = b3;
            for (int j = 0; j < H; j += 4) {
                const float4 h4 = *reinterpret_cast<const float4*>(hrow + j);
                t = __builtin_fmaf(A.w3[j], h4.x, t);
                t = __builtin_fmaf(A.w3[j + 1], h4.y, t);
                t = __builtin_fmaf(A.w3[j + 2], h4.z, t);
                t = __builtin_fmaf(A.w3[j + 3], h4.w, t);
            }
            A.scores[pp[lane]] = t;
        }
        wave_sync();
    }
}

hipError_t launch_rescore(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                          const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                          const int32_t* prompt_len, const int32_t* overlap, const int64_t* list,
                          const uint32_t* count, float* scores, int n_cu, hipStream_t s) {
    // the same chains as K=1 fp32 matrix-core steps (bit-identical), 32 candidates per wave
    if (m.mfma_chains && chain_mfma_supported(m))
        return launch_score_chain_mfma(m, compute, mu, inv_sigma, part_t, R, N, req_off, prompt_len, overlap, list,
                                       count, n_cu, scores, s);
    PairModel M{compute + m.c_w1, compute + m.c_w2t, compute + m.c_b2, compute + m.c_w3, compute + m.c_b3,
                m.d, m.d_inst, m.h1, m.h2};
    if (m.bf16 && m.h1 == m.h2 && (m.h1 == 64 || m.h1 == 128 || m.h1 == 256)) {
        RescoreArgs A{compute + m.c_w1, compute + m.c_w2t, compute + m.c_b2, compute + m.c_w3, compute + m.c_b3,
                      mu, inv_sigma, part_t, req_off, prompt_len, overlap, list, count, scores, N, m.d, m.d_inst,
                      m.block_tokens};
        const dim3 grid((uint32_t)n_cu), block(64 * kRescoreWaves);
        switch (m.h1) {
            case 64: hipLaunchKernelGGL(rescore_wave_kernel<64>, grid, block, 0, s, A); break;
            case 128: hipLaunchKernelGGL(rescore_wave_kernel<128>, grid, block, 0, s, A); break;
            default: hipLaunchKernelGGL(rescore_wave_kernel<256>, grid, block, 0, s, A); break;
        }
        return hipGetLastError();
    }
    // enough lanes for about two candidates per request, capped at 8 waves per SIMD
    int64_t want = ((int64_t)R * 2 + 255) / 256;
    int64_t cap = (int64_t)n_cu * 8;
    int64_t grid = want < cap ? want : cap;
    if (grid < 1) grid = 1;
    if (m.bf16)
        hipLaunchKernelGGL(rescore_kernel<true>, dim3((uint32_t)grid), dim3(256), 0, s, M, mu, inv_sigma, part_t, N,
                           req_off, prompt_len, overlap, m.block_tokens, list, count, scores);
    else
        hipLaunchKernelGGL(rescore_kernel<false>, dim3((uint32_t)grid), dim3(256), 0, s, M, mu, inv_sigma, part_t, N,
                           req_off, prompt_len, overlap, m.block_tokens, list, count, scores);
    return hipGetLastError();
}

}  // namespace ls
