// Prefix-cache state build: one open-addressing hash table per instance.
//
// The gateway's prefix index (Section 4.2, Prefix KV cache tracker; Section 2
// notes gateways use radix trees or hash tables) only has to answer "is block
// hash h cached on instance i".  On the GPU that is a membership probe, so the
// index is a bucketed hash table per instance: a bucket is 8 keys (64 bytes),
// tables are sized to about half load, and a full bucket overflows into the
// next one (linear probing over buckets).  Insertion is one thread per input
// hash with a 64-bit compare-and-swap per slot; duplicates collapse because a
// thread that finds its own key in a slot stops.
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

__global__ void table_insert_kernel(uint64_t* __restrict__ keys, const int64_t* __restrict__ base,
                                    const uint32_t* __restrict__ nbuckets, uint32_t* __restrict__ flags,
                                    const int64_t* __restrict__ inst_off, int32_t n_inst,
                                    const uint64_t* __restrict__ hashes, int64_t total) {
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= total) return;
    // owning instance: the largest i with inst_off[i] <= t
    int32_t lo = 0, hi = n_inst;
    while (hi - lo > 1) {
        int32_t mid = (lo + hi) >> 1;
        if (inst_off[mid] <= t) lo = mid; else hi = mid;
    }
    const int32_t i = lo;
    const uint64_t key = hashes[t];
    if (key == kEmptyKey) {
        atomicOr(&flags[i], kFlagHasEmptyKey);
        return;
    }
    const uint32_t nb = nbuckets[i];
    uint64_t* table = keys + base[i] * kBucketKeys;
    uint32_t b = bucket_of(key, nb);
    for (uint32_t probe = 0; probe < nb; ++probe) {
        uint64_t* bk = table + (int64_t)b * kBucketKeys;
        // read the whole bucket (one 64-byte line), then try its slots in order.
        // A slot changes at most once (empty -> key), so a stale read can only
        // show a filled slot as empty; the CAS on it then returns the key that
        // holds it.  Each slot is tried at most once per bucket, so the loop ends.
        const ulonglong2* q = reinterpret_cast<const ulonglong2*>(bk);
        const ulonglong2 v0 = q[0], v1 = q[1], v2 = q[2], v3 = q[3];
        const uint64_t slot[kBucketKeys] = {v0.x, v0.y, v1.x, v1.y, v2.x, v2.y, v3.x, v3.y};
#pragma unroll
        for (int s = 0; s < kBucketKeys; ++s) {
            if (slot[s] == key) return;
            if (slot[s] == kEmptyKey) {
                const unsigned long long old = atomicCAS((unsigned long long*)(bk + s), (unsigned long long)kEmptyKey,
                                                         (unsigned long long)key);
                if (old == kEmptyKey || old == key) return;
            }
        }
        b = (b + 1 == nb) ? 0 : b + 1;                 // bucket full without the key
    }
}

hipError_t launch_table_insert(const CacheTables& t, const int64_t* inst_off, const uint64_t* hashes,
                               int64_t total, int32_t n_inst, hipStream_t s) {
    if (total <= 0) return hipSuccess;
    const int block = 256;
    int64_t grid = (total + block - 1) / block;
    hipLaunchKernelGGL(table_insert_kernel, dim3((uint32_t)grid), dim3(block), 0, s, t.keys, t.base, t.nbuckets,
                       t.flags, inst_off, n_inst, hashes, total);
    return hipGetLastError();
}

}  // namespace ls
