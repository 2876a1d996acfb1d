// K1: prefix overlap of every (request, instance) pair.
//
// Prefix reuse is strictly sequential (Section 2, Background): a cached block
// counts only when every earlier block of the prompt is cached too, so the
// overlap l[r,i] is the length of the leading run of request r's block hashes
// that are members of instance i's cached set (Section 4.2, Prefix KV cache
// tracker: prompt in, expected hit per instance out).
//
// Requests that share a prompt prefix share the answer on that prefix.  The
// batch is grouped by first block hash; the longest request of each group is
// its leader and is probed in full.  Every other request r knows c, the length
// of its common prefix with the leader, and for each instance
//     l[r,i] = l[lead,i]                      if l[lead,i] < c
//     l[r,i] = c + (run of r from block c)    otherwise
// which is exact for any input (the first c blocks of r are the leader's), and
// turns the many repeated probes of a shared prefix into one.
//
// Probing.  Four lanes share one 64-byte bucket (16 bytes each), so a wave
// probes 16 pairs at once and every probe is one coalesced 64-byte read.  A
// group walks its request's blocks in order and speculatively probes a window
// of consecutive positions that doubles after every all-hit window (1, 2, 4,
// ... kMaxWindow): short runs waste few probes, long runs keep kMaxWindow reads
// in flight.  The first miss ends the pair.
#include "ls_internal.h"

namespace ls {

constexpr int kMaxWindow = 8;

// Extends a run that is known to hold for blocks [0, l) of h[0, n) on one table.
// All four lanes of a group call it together (it uses group-wide ballots).
__device__ __forceinline__ int64_t extend_run(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                              const uint64_t* __restrict__ h, int64_t n, int64_t l, int q, int shift) {
    int window = 1;
    while (l < n) {
        uint64_t key[kMaxWindow];
        ulonglong2 v[kMaxWindow];
        uint32_t bkt[kMaxWindow];
#pragma unroll
        for (int t = 0; t < kMaxWindow; ++t) {
            if (t < window && l + t < n) {
                key[t] = h[l + t];
                bkt[t] = bucket_of(key[t], nb);
                v[t] = *reinterpret_cast<const ulonglong2*>(table + (int64_t)bkt[t] * kBucketKeys + q * 2);
            }
        }
        bool stop = false;
#pragma unroll
        for (int t = 0; t < kMaxWindow; ++t) {
            if (!stop && t < window && l + t < n) {
                bool hit;
                if (key[t] == kEmptyKey) {
                    hit = has_empty;
                } else {
                    const uint64_t kk = key[t];
                    bool found = (v[t].x == kk) | (v[t].y == kk);
                    bool empty = (v[t].x == kEmptyKey) | (v[t].y == kEmptyKey);
                    bool gfound = ((__ballot(found) >> shift) & 0xFull) != 0;
                    bool gempty = ((__ballot(empty) >> shift) & 0xFull) != 0;
                    // bucket full without the key: it may have overflowed into the next buckets
                    uint32_t b = bkt[t];
                    for (uint32_t probe = 1; !gfound && !gempty && probe < nb; ++probe) {
                        b = (b + 1 == nb) ? 0 : b + 1;
                        const ulonglong2 w = *reinterpret_cast<const ulonglong2*>(table + (int64_t)b * kBucketKeys + q * 2);
                        found = (w.x == kk) | (w.y == kk);
                        empty = (w.x == kEmptyKey) | (w.y == kEmptyKey);
                        gfound = ((__ballot(found) >> shift) & 0xFull) != 0;
                        gempty = ((__ballot(empty) >> shift) & 0xFull) != 0;
                    }
                    hit = gfound;
                }
                if (hit) ++l;
                else stop = true;
            }
        }
        if (stop) break;
        window = window * 2 > kMaxWindow ? kMaxWindow : window * 2;
    }
    return l;
}

// ---------------------------------------------------------------------------
// grouping by first block hash
// ---------------------------------------------------------------------------
// slot of request r in the group table (-1: ungrouped, r leads itself); the
// group's leader word keeps max over members of (n_r << 32 | ~r): longest
// prompt, lowest id on ties.
__global__ void group_insert_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                    const uint64_t* __restrict__ req_hashes, uint64_t* __restrict__ gkeys,
                                    unsigned long long* __restrict__ glead, uint32_t G, int32_t* __restrict__ slot_of) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= R) return;
    const int64_t n = req_off[r + 1] - req_off[r];
    int32_t slot = -1;
    if (n > 0) {
        const uint64_t key = req_hashes[req_off[r]];
        if (key != kEmptyKey) {
            uint32_t b = bucket_of(key, G);
            for (uint32_t probe = 0; probe < G; ++probe) {
                const uint64_t cur = gkeys[b];
                if (cur == key) { slot = (int32_t)b; break; }
                if (cur == kEmptyKey) {
                    const unsigned long long old = atomicCAS((unsigned long long*)(gkeys + b),
                                                             (unsigned long long)kEmptyKey, (unsigned long long)key);
                    if (old == kEmptyKey || old == key) { slot = (int32_t)b; break; }
                }
                b = (b + 1 == G) ? 0 : b + 1;
            }
        }
    }
    slot_of[r] = slot;
    if (slot >= 0) {
        const unsigned long long word = ((unsigned long long)n << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)r);
        if (glead[slot] < word) atomicMax(glead + slot, word);
    }
}

// One wave per request: leader id and common-prefix length with the leader;
// leaders append themselves to the leader list.
__global__ __launch_bounds__(256) void group_lcp_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                                        const uint64_t* __restrict__ req_hashes,
                                                        const unsigned long long* __restrict__ glead,
                                                        const int32_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ lead_of, int32_t* __restrict__ lcp_of,
                                                        int32_t* __restrict__ leaders, uint32_t* __restrict__ n_leaders) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (r >= R) return;
    const int32_t slot = slot_of[r];
    const int64_t lead = slot < 0 ? r : (int64_t)(0xFFFFFFFFu - (uint32_t)(glead[slot] & 0xFFFFFFFFull));
    const int64_t n = req_off[r + 1] - req_off[r];
    int64_t c = n;
    if (lead != r) {
        const uint64_t* __restrict__ a = req_hashes + req_off[r];
        const uint64_t* __restrict__ b = req_hashes + req_off[lead];
        const int64_t nl = req_off[lead + 1] - req_off[lead];
        const int64_t m = n < nl ? n : nl;
        c = m;
        for (int64_t j0 = 0; j0 < m; j0 += 64) {
            const int64_t j = j0 + lane;
            const bool diff = j < m && a[j] != b[j];
            const uint64_t mask = __ballot(diff);
            if (mask) {
                c = j0 + __ffsll((long long)mask) - 1;
                break;
            }
        }
    }
    if (lane == 0) {
        lead_of[r] = (int32_t)lead;
        lcp_of[r] = (int32_t)c;
        if (lead == r) leaders[atomicAdd(n_leaders, 1u)] = (int32_t)r;
    }
}

// ---------------------------------------------------------------------------
// overlap kernels: leaders in full, then everyone from the leader's answer
// ---------------------------------------------------------------------------
struct ProbeTables {
    const uint64_t* __restrict__ keys;
    const int64_t* __restrict__ base;
    const uint32_t* __restrict__ nb;
    const uint32_t* __restrict__ flags;
};

__global__ __launch_bounds__(256) void prefix_leaders_kernel(ProbeTables T, int32_t N,
                                                             const int64_t* __restrict__ req_off,
                                                             const uint64_t* __restrict__ req_hashes,
                                                             const int32_t* __restrict__ leaders,
                                                             const uint32_t* __restrict__ n_leaders,
                                                             int32_t* __restrict__ overlap) {
    const int lane = threadIdx.x & 63;
    const int group = lane >> 2, q = lane & 3, shift = group * 4;
    const int64_t total = (int64_t)(*n_leaders) * N;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); w * 16 < total; w += waves) {
        const int64_t pair = w * 16 + group;
        if (pair >= total) continue;                     // whole group of 4 lanes skips together
        const int64_t k = pair / N, i = pair - k * N;
        const int64_t r = leaders[k];
        const int64_t h0 = req_off[r], n = req_off[r + 1] - h0;
        const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
        const int64_t l = extend_run(table, T.nb[i], (T.flags[i] & kFlagHasEmptyKey) != 0, req_hashes + h0, n, 0, q,
                                     shift);
        if (q == 0) overlap[r * N + i] = (int32_t)l;
    }
}

__global__ __launch_bounds__(256) void prefix_followers_kernel(ProbeTables T, int32_t R, int32_t N,
                                                               const int64_t* __restrict__ req_off,
                                                               const uint64_t* __restrict__ req_hashes,
                                                               const int32_t* __restrict__ lead_of,
                                                               const int32_t* __restrict__ lcp_of,
                                                               int32_t* __restrict__ overlap) {
    const int lane = threadIdx.x & 63;
    const int group = lane >> 2, q = lane & 3, shift = group * 4;
    const int64_t pair = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 16 + group;
    if (pair >= (int64_t)R * N) return;
    const int64_t r = pair / N, i = pair - r * N;
    const int64_t lead = lead_of[r];
    if (lead == r) return;                                // written by the leader pass
    const int64_t c = lcp_of[r];
    const int32_t ll = overlap[lead * N + i];
    int64_t l;
    if (ll < c) {
        l = ll;
    } else {
        const int64_t h0 = req_off[r], n = req_off[r + 1] - h0;
        const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
        l = extend_run(table, T.nb[i], (T.flags[i] & kFlagHasEmptyKey) != 0, req_hashes + h0, n, c, q, shift);
    }
    if (q == 0) overlap[pair] = (int32_t)l;
}

int64_t prefix_workspace_bytes(int32_t R) {
    const int64_t G = group_table_size(R);
    return G * 8 + G * 8 + (int64_t)R * 4 * 4 + 256;
}

hipError_t launch_prefix_match(const CacheTables& t, int32_t R, int32_t N, const int64_t* req_off,
                               const uint64_t* req_hashes, int32_t* overlap, void* workspace, int n_cu,
                               hipStream_t s) {
    const int64_t pairs = (int64_t)R * N;
    if (pairs <= 0) return hipSuccess;
    const int64_t G = group_table_size(R);
    char* p = reinterpret_cast<char*>(workspace);
    uint64_t* gkeys = reinterpret_cast<uint64_t*>(p); p += G * 8;
    unsigned long long* glead = reinterpret_cast<unsigned long long*>(p); p += G * 8;
    int32_t* slot_of = reinterpret_cast<int32_t*>(p); p += (int64_t)R * 4;
    int32_t* lead_of = reinterpret_cast<int32_t*>(p); p += (int64_t)R * 4;
    int32_t* lcp_of = reinterpret_cast<int32_t*>(p); p += (int64_t)R * 4;
    int32_t* leaders = reinterpret_cast<int32_t*>(p); p += (int64_t)R * 4;
    uint32_t* n_leaders = reinterpret_cast<uint32_t*>(p);

    hipError_t e = launch_fill_u64(gkeys, kEmptyKey, G, s);
    if (e == hipSuccess) e = launch_fill_u64(reinterpret_cast<uint64_t*>(glead), 0ull, G, s);
    if (e == hipSuccess) e = launch_fill_u32(n_leaders, 0u, 1, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(group_insert_kernel, dim3((uint32_t)(((int64_t)R + 255) / 256)), dim3(256), 0, s, R, req_off,
                       req_hashes, gkeys, glead, (uint32_t)G, slot_of);
    hipLaunchKernelGGL(group_lcp_kernel, dim3((uint32_t)(((int64_t)R + 3) / 4)), dim3(256), 0, s, R, req_off,
                       req_hashes, glead, slot_of, lead_of, lcp_of, leaders, n_leaders);
    ProbeTables T{t.keys, t.base, t.nbuckets, t.flags};
    // leaders: persistent grid over (leader, instance) pairs
    int64_t lgrid = (pairs + 63) / 64;
    const int64_t cap = (int64_t)n_cu * 32;
    if (lgrid > cap) lgrid = cap;
    hipLaunchKernelGGL(prefix_leaders_kernel, dim3((uint32_t)lgrid), dim3(256), 0, s, T, N, req_off, req_hashes,
                       leaders, n_leaders, overlap);
    hipLaunchKernelGGL(prefix_followers_kernel, dim3((uint32_t)((pairs + 63) / 64)), dim3(256), 0, s, T, R, N, req_off,
                       req_hashes, lead_of, lcp_of, overlap);
    return hipGetLastError();
}

}  // namespace ls
