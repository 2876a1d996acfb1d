// K1: prefix overlap of every (request, instance) pair.
//
// Prefix reuse is strictly sequential (Section 2, Background): a cached block
// counts only when every earlier block of the prompt is cached too, so the
// overlap l[r,i] is the length of the leading run of request r's block hashes
// that are members of instance i's cached set (Section 4.2, Prefix KV cache
// tracker: prompt in, expected hit per instance out).
//
// Mapping.  Four lanes share one 64-byte bucket (16 bytes each), so a wave
// probes 16 pairs at once and every probe is one coalesced 64-byte read.  A
// group walks its request's blocks in order; to hide the latency of those
// dependent reads it speculatively probes a window of consecutive positions
// that doubles after every all-hit window (1, 2, 4, ... kMaxWindow), so short
// runs waste at most a few probes and long runs keep kMaxWindow reads in
// flight per pair.  The first miss ends the pair.
#include "ls_internal.h"

namespace ls {

template <int kMaxWindow>
__global__ __launch_bounds__(256) void prefix_match_kernel(
    const uint64_t* __restrict__ keys, const int64_t* __restrict__ tbase, const uint32_t* __restrict__ tnb,
    const uint32_t* __restrict__ tflags, int32_t R, int32_t N, const int64_t* __restrict__ req_off,
    const uint64_t* __restrict__ req_hashes, int32_t* __restrict__ overlap) {
    const int lane = threadIdx.x & 63;
    const int group = lane >> 2;          // 16 groups per wave
    const int q = lane & 3;               // 16-byte quarter of the bucket
    const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const int64_t pair = wave * 16 + group;
    const int64_t total = (int64_t)R * N;
    const bool valid = pair < total;

    int64_t r = 0, i = 0;
    if (valid) {
        r = pair / N;
        i = pair - r * N;
    }
    const int64_t h0 = valid ? req_off[r] : 0;
    const int64_t n = valid ? req_off[r + 1] - h0 : 0;
    const uint64_t* __restrict__ h = req_hashes + h0;
    const uint32_t nb = valid ? tnb[i] : 1u;
    const uint64_t* __restrict__ table = keys + (valid ? tbase[i] : 0) * kBucketKeys;
    const bool has_empty = valid && (tflags[i] & kFlagHasEmptyKey);
    const int shift = group * 4;

    int64_t l = 0;
    bool done = !valid || n <= 0;
    int window = 1;
    while (!done) {
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
                    uint64_t kk = key[t];
                    bool found = (v[t].x == kk) | (v[t].y == kk);
                    bool empty = (v[t].x == kEmptyKey) | (v[t].y == kEmptyKey);
                    bool gfound = ((__ballot(found) >> shift) & 0xFull) != 0;
                    bool gempty = ((__ballot(empty) >> shift) & 0xFull) != 0;
                    // bucket full without the key: the key may have overflowed
                    // into the following buckets (rare at half load)
                    uint32_t b = bkt[t];
                    for (uint32_t probe = 1; !gfound && !gempty && probe < nb; ++probe) {
                        b = (b + 1 == nb) ? 0 : b + 1;
                        ulonglong2 w = *reinterpret_cast<const ulonglong2*>(table + (int64_t)b * kBucketKeys + q * 2);
                        found = (w.x == kk) | (w.y == kk);
                        empty = (w.x == kEmptyKey) | (w.y == kEmptyKey);
                        gfound = ((__ballot(found) >> shift) & 0xFull) != 0;
                        gempty = ((__ballot(empty) >> shift) & 0xFull) != 0;
                    }
                    hit = gfound;
                }
                if (hit) {
                    ++l;
                } else {
                    stop = true;
                }
            }
        }
        if (stop || l >= n) {
            done = true;
        } else {
            window = window * 2 > kMaxWindow ? kMaxWindow : window * 2;
        }
    }
    if (valid && q == 0) overlap[pair] = (int32_t)l;
}

hipError_t launch_prefix_match(const CacheTables& t, int32_t R, int32_t N, const int64_t* req_off,
                               const uint64_t* req_hashes, int32_t* overlap, hipStream_t s) {
    const int64_t pairs = (int64_t)R * N;
    if (pairs <= 0) return hipSuccess;
    const int block = 256;                           // 4 waves x 16 pairs
    const int64_t grid = (pairs + 63) / 64;
    hipLaunchKernelGGL(prefix_match_kernel<8>, dim3((uint32_t)grid), dim3(block), 0, s, t.keys, t.base, t.nbuckets,
                       t.flags, R, N, req_off, req_hashes, overlap);
    return hipGetLastError();
}

}  // namespace ls
