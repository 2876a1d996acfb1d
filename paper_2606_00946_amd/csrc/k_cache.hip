// Prefix-cache state build: one open-addressing hash table per instance.
//
// The gateway's prefix index (Section 4.2, Prefix KV cache tracker; Section 2
// notes gateways use radix trees or hash tables) only has to answer "is block
// hash h cached on instance i".  On the GPU that is a membership probe, so the
// index is a bucketed hash table per instance: a bucket is 8 keys (64 bytes),
// tables are sized to about half load, and a full bucket overflows into the
// next one (linear probing over buckets, wrapping at the table's end).  A
// lookup stops at the first bucket that holds the key or an empty slot.
//
// Build.  Random 64-bit compare-and-swaps on an HBM-resident table move whole
// cache lines in and out for every key, so the table is built in LDS instead:
// one workgroup owns a segment of kSegBuckets consecutive buckets of one
// instance (128 KiB), scans that instance's keys, and places the ones whose
// home bucket lies in its segment.  A slot is claimed with one LDS add on the
// bucket's fill counter (slots fill in order 0..7; a full bucket sends the key
// on to the next one) and written with one store; the finished segment goes
// out with coalesced stores.  A key whose probe runs past the segment's last
// bucket is queued and placed by a second, global pass that continues the
// probe from the next segment (rare at half load).  Either way every bucket
// between a key's home and its slot is full and the slots before it in its
// bucket are filled, which is all a lookup relies on.  Repeated input keys may
// each take a slot; the table is sized by the input count, so they still fit.
// Optionally the build records, for every slot it fills, the input position of
// the key placed there (`entry_of`), and per instance the position of the
// all-ones key (`eidx`): with unique keys per instance that is the slot map the
// index maintenance keeps.
#include "ls_internal.h"

namespace ls {

__global__ void fill_u64_kernel(uint64_t* __restrict__ p, uint64_t v, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

__global__ void fill_u32_kernel(uint32_t* __restrict__ p, uint32_t v, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

static int grid_for(int64_t n, int block) {
    int64_t g = (n + block - 1) / block;
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_fill_u64(uint64_t* p, uint64_t value, int64_t count, hipStream_t s) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(count, 256)), dim3(256), 0, s, p, value, count);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t count, hipStream_t s) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(count, 256)), dim3(256), 0, s, p, value, count);
    return hipGetLastError();
}

// Insert `key` into the table of nb buckets, probing from bucket b; returns the
// slot (bucket * 8 + position) that holds it, or -1 if the table is full.  A
// slot changes at most once (empty -> key), so a stale read can only show a
// filled slot as empty; the CAS on it then returns the key that holds it.
// Each slot is tried at most once per bucket, so the loop ends.
__device__ int64_t global_insert(uint64_t* table, uint32_t nb, uint32_t b, uint64_t key) {
    for (uint32_t probe = 0; probe < nb; ++probe) {
        uint64_t* bk = table + (int64_t)b * kBucketKeys;
        const ulonglong2* q = reinterpret_cast<const ulonglong2*>(bk);
        const ulonglong2 v0 = q[0], v1 = q[1], v2 = q[2], v3 = q[3];
        const uint64_t slot[kBucketKeys] = {v0.x, v0.y, v1.x, v1.y, v2.x, v2.y, v3.x, v3.y};
#pragma unroll
        for (int s = 0; s < kBucketKeys; ++s) {
            if (slot[s] == key) return (int64_t)b * kBucketKeys + s;
            if (slot[s] == kEmptyKey) {
                const unsigned long long old = atomicCAS((unsigned long long*)(bk + s), (unsigned long long)kEmptyKey,
                                                         (unsigned long long)key);
                if (old == kEmptyKey || old == key) return (int64_t)b * kBucketKeys + s;
            }
        }
        b = (b + 1 == nb) ? 0 : b + 1;                 // bucket full without the key
    }
    return -1;
}

// Place `key` in an LDS segment of nbl buckets, probing from local bucket lb:
// the bucket's fill counter hands out slots in order.  Returns the local slot,
// or -1 when the probe runs past the segment's last bucket.
__device__ __forceinline__ int32_t segment_place(uint64_t* seg, uint32_t* fill, uint32_t lb, uint32_t nbl,
                                                 uint64_t key) {
    for (; lb < nbl; ++lb) {
        const uint32_t slot = atomicAdd(&fill[lb], 1u);
        if (slot < (uint32_t)kBucketKeys) {
            seg[lb * kBucketKeys + slot] = key;
            return (int32_t)(lb * kBucketKeys + slot);
        }
    }
    return -1;
}

__device__ __forceinline__ int32_t owner_of(const int64_t* __restrict__ off, int32_t n, int64_t t) {
    // the largest i in [0, n) with off[i] <= t
    int32_t lo = 0, hi = n;
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (off[mid] <= t) lo = mid; else hi = mid;
    }
    return lo;
}

constexpr int kSegThreads = 1024;

__global__ __launch_bounds__(kSegThreads) void table_segment_kernel(
    uint64_t* __restrict__ keys, const int64_t* __restrict__ base, const uint32_t* __restrict__ nbuckets,
    uint32_t* __restrict__ flags, const int64_t* __restrict__ inst_off, const int32_t* __restrict__ seg_off,
    int32_t n_inst, const uint64_t* __restrict__ hashes, int64_t* __restrict__ ovf, uint32_t* __restrict__ ovf_count,
    uint32_t ovf_cap, uint32_t* __restrict__ entry_of, int64_t* __restrict__ eidx) {
    __shared__ uint64_t seg[kSegBuckets * kBucketKeys];
    __shared__ uint32_t fill[kSegBuckets];
    // Workgroups are dealt to the 8 XCDs round-robin; renumber them so that the
    // segments of one instance run on one XCD and share its L2 copy of the keys.
    const uint32_t G = gridDim.x, G8 = G / 8, w = blockIdx.x;
    const uint32_t L = (w < G8 * 8) ? (w % 8) * G8 + w / 8 : w;
    int32_t lo = 0, hi = n_inst;                    // the instance: largest i with seg_off[i] <= L
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if ((uint32_t)seg_off[mid] <= L) lo = mid; else hi = mid;
    }
    const int32_t i = lo;
    const uint32_t s = L - (uint32_t)seg_off[i];
    const uint32_t nb = nbuckets[i];
    const uint32_t b0 = s * kSegBuckets;
    const uint32_t nbl = min((uint32_t)kSegBuckets, nb - b0);
    const int tid = threadIdx.x;

    ulonglong2* seg2 = reinterpret_cast<ulonglong2*>(seg);
    const ulonglong2 empty2 = {kEmptyKey, kEmptyKey};
    for (uint32_t x = tid; x < nbl * (kBucketKeys / 2); x += kSegThreads) seg2[x] = empty2;
    for (uint32_t x = tid; x < nbl; x += kSegThreads) fill[x] = 0u;
    __syncthreads();

    const int64_t t0 = inst_off[i], t1 = inst_off[i + 1];
    int has_empty = 0;
    for (int64_t t = t0 + tid; t < t1; t += 4 * kSegThreads) {
        uint64_t k[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) k[u] = (t + u * kSegThreads < t1) ? hashes[t + u * kSegThreads] : kEmptyKey;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (t + u * kSegThreads >= t1) continue;
            if (k[u] == kEmptyKey) {
                has_empty = 1;
                if (eidx) eidx[i] = t + u * kSegThreads;
                continue;
            }
            const uint32_t lb = bucket_of(k[u], nb) - b0;
            if (lb >= nbl) continue;                // home bucket in another segment
            const int32_t ls = segment_place(seg, fill, lb, nbl, k[u]);
            if (ls < 0) {
                const uint32_t pos = atomicAdd(ovf_count, 1u);
                if (pos < ovf_cap) ovf[pos] = t + u * kSegThreads;
            } else if (entry_of) {
                entry_of[(base[i] + b0) * kBucketKeys + ls] = (uint32_t)(t + u * kSegThreads);
            }
        }
    }
    has_empty = __syncthreads_or(has_empty);
    if (s == 0 && tid == 0) flags[i] = has_empty ? kFlagHasEmptyKey : 0u;
    // streaming stores: the finished segment is not read again by this build,
    // and keeping it out of L2 leaves room for the keys the instance's other
    // segments are still scanning
    ulonglong2* dst = reinterpret_cast<ulonglong2*>(keys + (base[i] + b0) * kBucketKeys);
    for (uint32_t x = tid; x < nbl * (kBucketKeys / 2); x += kSegThreads) {
        const ulonglong2 v = seg2[x];
        __builtin_nontemporal_store(v.x, &dst[x].x);
        __builtin_nontemporal_store(v.y, &dst[x].y);
    }
}

// Keys whose probe ran past their segment continue in the next segment.  If
// more keys overflowed than the queue holds, every key is (re)inserted from
// its home bucket instead: keys already placed are found on their probe path,
// so that is correct too, only slower.
__global__ void table_overflow_kernel(uint64_t* __restrict__ keys, const int64_t* __restrict__ base,
                                      const uint32_t* __restrict__ nbuckets, const int64_t* __restrict__ inst_off,
                                      int32_t n_inst, const uint64_t* __restrict__ hashes, int64_t total,
                                      const int64_t* __restrict__ ovf, const uint32_t* __restrict__ ovf_count,
                                      uint32_t ovf_cap, uint32_t* __restrict__ entry_of) {
    const uint32_t n = *ovf_count;
    if (n == 0) return;
    const bool queued = n <= ovf_cap;
    const int64_t n_keys = inst_off[n_inst] < total ? inst_off[n_inst] : total;   // total bounds the key count
    const int64_t count = queued ? (int64_t)n : n_keys;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < count; j += stride) {
        const int64_t t = queued ? ovf[j] : j;
        const uint64_t key = hashes[t];
        if (key == kEmptyKey) continue;
        const int32_t i = owner_of(inst_off, n_inst, t);
        const uint32_t nb = nbuckets[i];
        uint32_t b = bucket_of(key, nb);
        if (queued) {
            b = (b / kSegBuckets + 1) * kSegBuckets;
            if (b >= nb) b = 0;
        }
        const int64_t q = global_insert(keys + base[i] * kBucketKeys, nb, b, key);
        if (entry_of && q >= 0) entry_of[base[i] * kBucketKeys + q] = (uint32_t)t;
    }
}

int64_t table_overflow_capacity(int64_t total) { return 4096 + total / 64; }

hipError_t launch_table_build(const CacheTables& t, const int64_t* inst_off, const int32_t* seg_off, int32_t n_seg,
                              const uint64_t* hashes, int64_t total, int32_t n_inst, void* ovf_ws, int n_cu,
                              hipStream_t s, uint32_t* entry_of, int64_t* eidx) {
    uint32_t* count = reinterpret_cast<uint32_t*>(ovf_ws);
    int64_t* list = reinterpret_cast<int64_t*>(static_cast<char*>(ovf_ws) + 256);
    const uint32_t cap = (uint32_t)table_overflow_capacity(total);
    hipError_t e = launch_fill_u32(count, 0u, 1, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(table_segment_kernel, dim3((uint32_t)n_seg), dim3(kSegThreads), 0, s, t.keys, t.base,
                       t.nbuckets, t.flags, inst_off, seg_off, n_inst, hashes, list, count, cap, entry_of, eidx);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(table_overflow_kernel, dim3((uint32_t)(4 * n_cu)), dim3(256), 0, s, t.keys, t.base,
                       t.nbuckets, inst_off, n_inst, hashes, total, list, count, cap, entry_of);
    return hipGetLastError();
}

}  // namespace ls
