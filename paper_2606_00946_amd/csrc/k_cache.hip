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
// instance (128 KiB) and places the keys whose home bucket lies in it.  The
// keys reach their segment's workgroup through a partition: one pass computes
// every key's segment and appends the key, with its input position, to that
// segment's run (LDS histograms per chunk, one global add per segment
// touched).  A run holds as many keys as the segment has slots (the runs are
// laid out like the table's slots); keys past that could not all fit in the
// segment anyway and go straight to the global pass.
// Each key is thus read twice in all, instead of once by every segment of its
// instance.  A slot is claimed with one LDS add on the
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
// Every build also leaves a 32-bit fingerprint of each cached key, segment by
// segment, for the prefix pass: the segment workgroup writes its run's
// fingerprints with coalesced stores as it reads the run (4 bytes per key, a
// quarter of what the table's slots take), and the global pass lists those of
// the keys it inserts.
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

struct FillOps {
    FillOp op[kMaxFillOps];
};

// blockIdx.y = the fill
__global__ void fill_multi_kernel(FillOps F) {
    const FillOp o = F.op[blockIdx.y];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < o.count; i += stride) {
        if (o.bytes == 8) static_cast<uint64_t*>(o.p)[i] = o.value;
        else static_cast<uint32_t*>(o.p)[i] = (uint32_t)o.value;
    }
}

hipError_t launch_fill_multi(const FillOp* ops, int n, hipStream_t s) {
    if (n > kMaxFillOps) return hipErrorInvalidValue;
    FillOps F{};
    int m = 0;
    int64_t most = 0;
    for (int i = 0; i < n; ++i) {
        if (ops[i].count <= 0) continue;
        if (ops[i].bytes != 4 && ops[i].bytes != 8) return hipErrorInvalidValue;
        F.op[m++] = ops[i];
        most = ops[i].count > most ? ops[i].count : most;
    }
    if (m == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_multi_kernel, dim3(grid_for(most, 256), m), dim3(256), 0, s, F);
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
constexpr int kPartThreads = 1024;
constexpr int kPartPerThread = 8;              // consecutive keys per thread
constexpr int64_t kPartChunk = (int64_t)kPartThreads * kPartPerThread;
constexpr int kPartBins = 4096;                // LDS counters; wider segment ranges use global adds

constexpr int kPartInst = 1024;                // instances a chunk may span with its table in LDS

// Queue entry for a key that did not fit its segment's run: its position,
// complemented, so that the global pass probes from its home bucket (an entry
// that overflowed the segment itself is the position, probed from the next
// segment).
__device__ __forceinline__ void queue_overflow(int64_t t, bool from_home, int64_t* ovf, uint32_t* ovf_count,
                                               uint32_t ovf_cap) {
    const uint32_t pos = atomicAdd(ovf_count, 1u);
    if (pos < ovf_cap) ovf[pos] = from_home ? ~t : t;
}

// A build without a slot map keeps no input positions beside the runs: a key
// that overflows its segment is queued by its position q in the runs instead,
// as kRunPosTag + q, and probed from the next segment like a position entry.
constexpr int64_t kRunPosTag = (int64_t)1 << 62;

// Segment (global index) of every key of the chunk, and the key appended to
// that segment's run.  The workgroup first finds the instances its chunk spans
// (one parallel pass over the offsets) and copies their offsets, first
// segments and bucket counts to LDS; a thread then takes PER consecutive keys
// and walks the instance boundaries from its first key.  The all-ones key sets
// its instance's flag instead (and records its position in eidx).
//
// STAGE (builds without a slot map): the chunk's keys are first gathered in
// LDS ordered by segment (the counts' prefix sums plus each key's rank), then
// written out with consecutive threads on consecutive slots of each run, so
// the run writes are coalesced instead of one scattered 8-byte store per key.
// Every key lands in the slot the direct write would give it.
template <bool IDX, int PER, bool STAGE>
__global__ __launch_bounds__(kPartThreads) void part_kernel(const uint64_t* __restrict__ hashes,
                                                            const int64_t* __restrict__ inst_off,
                                                            const int32_t* __restrict__ seg_off,
                                                            const uint32_t* __restrict__ nbuckets,
                                                            const int64_t* __restrict__ base, int32_t n_inst,
                                                            int64_t total, uint32_t* __restrict__ seg_cursor,
                                                            uint64_t* __restrict__ part_key,
                                                            uint32_t* __restrict__ part_idx,
                                                            uint32_t* __restrict__ flags, int64_t* __restrict__ eidx,
                                                            int64_t* __restrict__ ovf, uint32_t* __restrict__ ovf_count,
                                                            uint32_t ovf_cap) {
    static_assert(!(STAGE && IDX), "staging keeps no input positions");
    constexpr int64_t CH = (int64_t)kPartThreads * PER;
    constexpr int BINS = STAGE ? kPartThreads : kPartBins;        // staging: one bin per thread for the scan
    __shared__ uint32_t bin[BINS];
    __shared__ int64_t l_off[kPartInst + 1];
    __shared__ int32_t l_seg[kPartInst + 1];
    __shared__ uint32_t l_nb[kPartInst];
    __shared__ int64_t l_base[kPartInst];
    __shared__ int32_t i_first, i_last;
    __shared__ uint64_t stage_k[STAGE ? CH : 1];                  // keys ordered by segment
    __shared__ uint16_t stage_s[STAGE ? CH : 1];                  // their local segment
    __shared__ uint32_t lofs[STAGE ? BINS : 1];                   // first staged slot of each local segment
    __shared__ uint32_t wsum[kPartThreads / 64];
    const int64_t n_keys = inst_off[n_inst] < total ? inst_off[n_inst] : total;
    const int64_t c0 = (int64_t)blockIdx.x * CH;
    if (c0 >= n_keys) return;                                     // uniform
    const int64_t c1 = c0 + CH < n_keys ? c0 + CH : n_keys;
    // the instances holding positions c0 and c1 - 1 (each owned by exactly one non-empty instance)
    for (int32_t i = threadIdx.x; i < n_inst; i += kPartThreads) {
        const int64_t a = inst_off[i], b = inst_off[i + 1];
        if (a <= c0 && c0 < b) i_first = i;
        if (a <= c1 - 1 && c1 - 1 < b) i_last = i;
    }
    for (int x = threadIdx.x; x < BINS; x += kPartThreads) bin[x] = 0u;
    __syncthreads();
    const int32_t ilo = i_first, ihi = i_last;
    const bool in_lds = ihi - ilo < kPartInst;
    if (in_lds) {
        for (int32_t x = threadIdx.x; x <= ihi - ilo + 1; x += kPartThreads) {
            l_off[x] = inst_off[ilo + x];
            l_seg[x] = seg_off[ilo + x];
            if (x <= ihi - ilo) {
                l_nb[x] = nbuckets[ilo + x];
                l_base[x] = base[ilo + x];
            }
        }
    }
    __syncthreads();
    const int32_t seg_lo = seg_off[ilo];
    const bool local = seg_off[ihi + 1] - seg_lo <= BINS;
    const int64_t t0 = c0 + (int64_t)threadIdx.x * PER;
    uint64_t key[PER];
    int32_t seg[PER];
    uint32_t rank[PER];
    int64_t run0[PER];                 // the segment's run: first slot and length in slots
    uint32_t runcap[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) key[u] = t0 + u < c1 ? hashes[t0 + u] : kEmptyKey;
    // instance of the first key, relative to ilo when the table is in LDS
    int32_t i = 0;
    if (t0 < c1) {
        if (in_lds) {
            int32_t lo = 0, hi = ihi - ilo + 1;                   // largest x with l_off[x] <= t0
            while (hi - lo > 1) {
                const int32_t mid = (lo + hi) >> 1;
                if (l_off[mid] <= t0) lo = mid; else hi = mid;
            }
            i = lo;
        } else {
            i = owner_of(inst_off, n_inst, t0);
        }
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int64_t t = t0 + u;
        seg[u] = -1;
        if (t >= c1) continue;
        int32_t first_seg;
        uint32_t nb;
        int64_t b_inst;
        if (in_lds) {
            while (l_off[i + 1] <= t) ++i;                       // empty instances are skipped too
            first_seg = l_seg[i];
            nb = l_nb[i];
            b_inst = l_base[i];
        } else {
            while (inst_off[i + 1] <= t) ++i;
            first_seg = seg_off[i];
            nb = nbuckets[i];
            b_inst = base[i];
        }
        if (key[u] == kEmptyKey) {
            const int32_t gi = in_lds ? ilo + i : i;
            atomicOr(&flags[gi], kFlagHasEmptyKey);
            if (eidx) eidx[gi] = t;
            continue;
        }
        const uint32_t sl = bucket_of(key[u], nb) / kSegBuckets;
        seg[u] = first_seg + (int32_t)sl;
        run0[u] = (b_inst + (int64_t)sl * kSegBuckets) * kBucketKeys;
        runcap[u] = min((uint32_t)kSegBuckets, nb - sl * kSegBuckets) * kBucketKeys;
        rank[u] = local ? atomicAdd(&bin[seg[u] - seg_lo], 1u) : 0u;
        if (!local) {
            const uint32_t pos = atomicAdd(&seg_cursor[seg[u]], 1u);
            if (pos < runcap[u]) {
                const int64_t q = run0[u] + pos;
                part_key[q] = key[u];
                if (IDX) part_idx[q] = (uint32_t)t;
            } else {
                queue_overflow(t, true, ovf, ovf_count, ovf_cap);
            }
            seg[u] = -1;
        }
    }
    if (!local) return;                                           // uniform
    __syncthreads();
    const int32_t nb_local = seg_off[ihi + 1] - seg_lo;
    // staging reads the instances' segments from LDS: only when they are there
    if (STAGE && in_lds) {                                        // uniform
        // exclusive prefix sum of the counts, one bin per thread (wave scans,
        // then the waves' totals)
        const int x = (int)threadIdx.x, lane = x & 63, wv = x >> 6;
        const uint32_t cnt = x < nb_local ? bin[x] : 0u;
        uint32_t v = cnt;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t y = __shfl_up(v, off);
            if (lane >= off) v += y;
        }
        if (lane == 63) wsum[wv] = v;
        __syncthreads();
        if (wv == 0) {
            uint32_t w = lane < kPartThreads / 64 ? wsum[lane] : 0u;
#pragma unroll
            for (int off = 1; off < kPartThreads / 64; off <<= 1) {
                const uint32_t y = __shfl_up(w, off);
                if (lane >= off) w += y;
            }
            if (lane < kPartThreads / 64) wsum[lane] = w;
        }
        __syncthreads();
        const uint32_t staged = wsum[kPartThreads / 64 - 1];
        if (x < nb_local) {
            lofs[x] = (wv ? wsum[wv - 1] : 0u) + v - cnt;
            if (cnt != 0u) bin[x] = atomicAdd(&seg_cursor[seg_lo + x], cnt);   // this chunk's first position in the run
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            if (seg[u] < 0) continue;
            const int ls = seg[u] - seg_lo;
            const uint32_t at = lofs[ls] + rank[u];
            stage_s[at] = (uint16_t)ls;
            stage_k[at] = key[u];
            if (bin[ls] + rank[u] >= runcap[u]) queue_overflow(t0 + u, true, ovf, ovf_count, ovf_cap);
        }
        __syncthreads();
        for (uint32_t at = threadIdx.x; at < staged; at += kPartThreads) {
            const int ls = stage_s[at];
            const uint32_t pos = bin[ls] + (at - lofs[ls]);
            // the instance holding local segment ls: the last one whose segments start at or before it
            const int32_t g = seg_lo + ls;
            int32_t lo = 0, hi = ihi - ilo + 1;
            while (hi - lo > 1) {
                const int32_t mid = (lo + hi) >> 1;
                if (l_seg[mid] <= g) lo = mid; else hi = mid;
            }
            const uint32_t sl = (uint32_t)(g - l_seg[lo]);
            const uint32_t cap = min((uint32_t)kSegBuckets, l_nb[lo] - sl * kSegBuckets) * kBucketKeys;
            if (pos < cap) part_key[(l_base[lo] + (int64_t)sl * kSegBuckets) * kBucketKeys + pos] = stage_k[at];
        }
        return;
    }
    for (int x = threadIdx.x; x < nb_local; x += kPartThreads) {
        const uint32_t cnt = bin[x];
        if (cnt != 0u) bin[x] = atomicAdd(&seg_cursor[seg_lo + x], cnt);   // this chunk's first position in the run
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        if (seg[u] < 0) continue;
        const uint32_t pos = bin[seg[u] - seg_lo] + rank[u];
        if (pos < runcap[u]) {
            const int64_t q = run0[u] + pos;
            part_key[q] = key[u];
            if (IDX) part_idx[q] = (uint32_t)(t0 + u);
        } else {
            queue_overflow(t0 + u, true, ovf, ovf_count, ovf_cap);
        }
    }
}

// The instance of every segment, for the segment build.
__global__ void seg_inst_kernel(const int32_t* __restrict__ seg_off, int32_t n_inst, int32_t* __restrict__ seg_inst) {
    const int32_t i = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i >= n_inst) return;
    for (int32_t x = seg_off[i]; x < seg_off[i + 1]; ++x) seg_inst[x] = i;
}

__global__ __launch_bounds__(kSegThreads) void table_segment_kernel(
    uint64_t* __restrict__ keys, const int64_t* __restrict__ base, const uint32_t* __restrict__ nbuckets,
    const int32_t* __restrict__ seg_off, const int32_t* __restrict__ seg_inst, const uint32_t* __restrict__ run_len,
    const uint64_t* __restrict__ part_key, const uint32_t* __restrict__ part_idx, int64_t* __restrict__ ovf,
    uint32_t* __restrict__ ovf_count, uint32_t ovf_cap, uint32_t* __restrict__ entry_of, uint32_t* __restrict__ fp,
    uint32_t* __restrict__ fp_len, uint32_t* __restrict__ fp_inst) {
    __shared__ uint64_t seg[kSegBuckets * kBucketKeys];
    __shared__ uint32_t fill[kSegBuckets];
    const uint32_t L = blockIdx.x;
    const int32_t i = seg_inst[L];
    const uint32_t s = L - (uint32_t)seg_off[i];
    const uint32_t nb = nbuckets[i];
    const uint32_t b0 = s * kSegBuckets;
    const uint32_t nbl = min((uint32_t)kSegBuckets, nb - b0);
    const int tid = threadIdx.x;
    constexpr int SPT = (int)(kSegSlots / kSegThreads);           // run slots per thread
    static_assert(kSegSlots % kSegThreads == 0, "a run fills whole rounds of the workgroup");

    // the run, laid out like the segment's slots: every key of the thread is
    // loaded at once, before the segment is cleared
    const int64_t r0 = (base[i] + b0) * kBucketKeys;
    const uint32_t len = min(run_len[L], nbl * (uint32_t)kBucketKeys);
    uint64_t rk[SPT];
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
        const uint32_t o = (uint32_t)tid + (uint32_t)u * kSegThreads;
        rk[u] = o < len ? part_key[r0 + o] : kEmptyKey;
    }

    ulonglong2* seg2 = reinterpret_cast<ulonglong2*>(seg);
    const ulonglong2 empty2 = {kEmptyKey, kEmptyKey};
    for (uint32_t x = tid; x < nbl * (kBucketKeys / 2); x += kSegThreads) seg2[x] = empty2;
    for (uint32_t x = tid; x < nbl; x += kSegThreads) fill[x] = 0u;
    __syncthreads();

    uint32_t* __restrict__ fp_run = fp + (int64_t)L * kSegSlots;
    if (tid == 0) {
        fp_len[L] = len;
        fp_inst[L] = (uint32_t)i;
    }
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
        const uint32_t o = (uint32_t)tid + (uint32_t)u * kSegThreads;
        if (o >= len) continue;
        const int64_t q = r0 + o;
        const uint64_t key = rk[u];
        fp_run[o] = key_fp(key);             // every key of the run is cached, placed here or by the global pass
        const uint32_t lb = bucket_of(key, nb) - b0;
        const int32_t ls = segment_place(seg, fill, lb, nbl, key);
        if (ls < 0) {
            if (entry_of) {
                queue_overflow(part_idx[q], false, ovf, ovf_count, ovf_cap);
            } else {
                const uint32_t pos = atomicAdd(ovf_count, 1u);
                if (pos < ovf_cap) ovf[pos] = kRunPosTag + q;
            }
        } else if (entry_of) {
            entry_of[(base[i] + b0) * kBucketKeys + ls] = part_idx[q];
        }
    }
    __syncthreads();
    // streaming stores: the finished segment is not read again by this build
    ulonglong2* dst = reinterpret_cast<ulonglong2*>(keys + (base[i] + b0) * kBucketKeys);
    for (uint32_t x = tid; x < nbl * (kBucketKeys / 2); x += kSegThreads) {
        const ulonglong2 v = seg2[x];
        __builtin_nontemporal_store(v.x, &dst[x].x);
        __builtin_nontemporal_store(v.y, &dst[x].y);
    }
}

// Keys whose probe ran past their segment continue in the next segment; keys
// that did not fit their segment's run are inserted from their home bucket.
// If more keys overflowed than the queue holds, every key is (re)inserted from
// its home bucket instead: keys already placed are found on their probe path,
// so that is correct too, only slower.  The fingerprints of the queued keys go
// to fp_extra (entry j of the queue at j) and their count to fp_meta[0]; a full
// queue records a count above both capacities, as the keys past a run's end
// are then listed nowhere.
__global__ void table_overflow_kernel(uint64_t* __restrict__ keys, const int64_t* __restrict__ base,
                                      const uint32_t* __restrict__ nbuckets, const int64_t* __restrict__ inst_off,
                                      int32_t n_inst, const uint64_t* __restrict__ hashes, int64_t total,
                                      const uint64_t* __restrict__ part_key,
                                      const int64_t* __restrict__ ovf, const uint32_t* __restrict__ ovf_count,
                                      uint32_t ovf_cap, uint32_t* __restrict__ entry_of, uint32_t* __restrict__ fp_extra,
                                      uint32_t* __restrict__ fp_extra_inst, uint32_t fp_extra_cap,
                                      uint32_t* __restrict__ fp_meta) {
    const uint32_t n = *ovf_count;
    const bool queued = n <= ovf_cap;
    if (blockIdx.x == 0 && threadIdx.x == 0) fp_meta[0] = queued && n <= fp_extra_cap ? n : 0xFFFFFFFFu;
    if (n == 0) return;
    const int64_t n_keys = inst_off[n_inst] < total ? inst_off[n_inst] : total;   // total bounds the key count
    const int64_t count = queued ? (int64_t)n : n_keys;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < count; j += stride) {
        const int64_t entry = queued ? ovf[j] : j;
        uint64_t key;
        int32_t i;
        int64_t t = -1;                                   // input position, when the entry has one
        bool next_segment;
        if (queued && entry >= kRunPosTag) {              // overflowed its segment, queued by run position
            const int64_t q = entry - kRunPosTag;
            key = part_key[q];
            i = owner_of(base, n_inst, q / kBucketKeys);  // base[i]: instance i's first bucket, increasing
            next_segment = true;
        } else {
            const bool from_home = entry < 0;             // past its segment's run: probe from home
            t = from_home ? ~entry : entry;
            key = hashes[t];
            i = owner_of(inst_off, n_inst, t);
            next_segment = queued && !from_home;
        }
        if (queued && j < (int64_t)fp_extra_cap) {
            fp_extra[j] = key == kEmptyKey ? kFpEmpty : key_fp(key);
            fp_extra_inst[j] = (uint32_t)i;
        }
        if (key == kEmptyKey) continue;
        const uint32_t nb = nbuckets[i];
        uint32_t b = bucket_of(key, nb);
        if (next_segment) {
            b = (b / kSegBuckets + 1) * kSegBuckets;
            if (b >= nb) b = 0;
        }
        const int64_t q = global_insert(keys + base[i] * kBucketKeys, nb, b, key);
        if (entry_of && q >= 0 && t >= 0) entry_of[base[i] * kBucketKeys + q] = (uint32_t)t;
    }
}

int64_t table_overflow_capacity(int64_t total) { return 4096 + total / 64; }

static int64_t up256(int64_t b) { return (b + 255) / 256 * 256; }

int64_t table_fp_bytes(int32_t n_seg, int64_t extra_cap) {
    const int64_t segs = n_seg > 0 ? n_seg : 1, extra = extra_cap > 0 ? extra_cap : 1;
    return up256(4 * segs * kSegSlots) + 2 * up256(4 * segs) + 2 * up256(4 * extra) + 256;
}

void carve_table_fp(CacheTables& t, void* buf, int32_t n_seg, int64_t extra_cap) {
    char* p = static_cast<char*>(buf);
    const int64_t segs = n_seg > 0 ? n_seg : 1, extra = extra_cap > 0 ? extra_cap : 1;
    t.fp = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * segs * kSegSlots);
    t.fp_len = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * segs);
    t.fp_inst = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * segs);
    t.fp_extra = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * extra);
    t.fp_extra_inst = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * extra);
    t.fp_meta = reinterpret_cast<uint32_t*>(p);
    t.fp_extra_cap = extra_cap;
    t.n_seg = n_seg;
}

// Workspace: overflow counter (256 B) and queue, run lengths, the instance of
// every segment, and the runs: a key and input position per table slot.
struct BuildWs {
    uint32_t* ovf_count;
    int64_t* ovf;
    uint32_t* run_len;
    int32_t* seg_inst;
    uint64_t* part_key;
    uint32_t* part_idx;
};

static BuildWs carve_build_ws(void* ws, int64_t total, int32_t n_seg, int64_t total_buckets) {
    char* p = static_cast<char*>(ws);
    const int64_t runs = (total_buckets > 0 ? total_buckets : 1) * kBucketKeys;
    BuildWs w;
    w.ovf_count = reinterpret_cast<uint32_t*>(p);
    p += 256;
    w.ovf = reinterpret_cast<int64_t*>(p);
    p += up256(8 * table_overflow_capacity(total));
    w.run_len = reinterpret_cast<uint32_t*>(p);
    p += up256(4 * ((int64_t)n_seg + 1));
    w.seg_inst = reinterpret_cast<int32_t*>(p);
    p += up256(4 * ((int64_t)n_seg + 1));
    w.part_key = reinterpret_cast<uint64_t*>(p);
    p += up256(8 * runs);
    w.part_idx = reinterpret_cast<uint32_t*>(p);
    return w;
}

int64_t table_build_workspace_bytes(int64_t total, int32_t n_seg, int64_t total_buckets) {
    const int64_t runs = (total_buckets > 0 ? total_buckets : 1) * kBucketKeys;
    return 256 + up256(8 * table_overflow_capacity(total)) + 2 * up256(4 * ((int64_t)n_seg + 1)) + up256(8 * runs) +
           up256(4 * runs);
}

hipError_t launch_table_build(const CacheTables& t, const int64_t* inst_off, const int32_t* seg_off, int32_t n_seg,
                              const uint64_t* hashes, int64_t total, int32_t n_inst, void* ws, int n_cu,
                              hipStream_t s, uint32_t* entry_of, int64_t* eidx) {
    if (!t.fp || !t.fp_len || !t.fp_inst || !t.fp_extra || !t.fp_extra_inst || !t.fp_meta || t.n_seg < n_seg)
        return hipErrorInvalidValue;
    const BuildWs w = carve_build_ws(ws, total, n_seg, t.total_buckets);
    const uint32_t cap = (uint32_t)table_overflow_capacity(total);
    hipError_t e;
    const FillOp fills[3] = {{w.ovf_count, 0u, 1, 4}, {w.run_len, 0u, (int64_t)n_seg + 1, 4}, {t.flags, 0u, n_inst, 4}};
    if ((e = launch_fill_multi(fills, 3, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(seg_inst_kernel, dim3((uint32_t)((n_inst + 255) / 256)), dim3(256), 0, s, seg_off, n_inst,
                       w.seg_inst);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (total > 0) {
        // input positions beside the runs only for a slot map; otherwise the
        // runs are written through LDS staging, half-size chunks
        if (entry_of) {
            constexpr int64_t ch = kPartChunk;
            hipLaunchKernelGGL((part_kernel<true, kPartPerThread, false>), dim3((uint32_t)((total + ch - 1) / ch)),
                               dim3(kPartThreads), 0, s, hashes, inst_off, seg_off, t.nbuckets, t.base, n_inst, total,
                               w.run_len, w.part_key, w.part_idx, t.flags, eidx, w.ovf, w.ovf_count, cap);
        } else {
            constexpr int64_t ch = (int64_t)kPartThreads * (kPartPerThread / 2);
            hipLaunchKernelGGL((part_kernel<false, kPartPerThread / 2, true>), dim3((uint32_t)((total + ch - 1) / ch)),
                               dim3(kPartThreads), 0, s, hashes, inst_off, seg_off, t.nbuckets, t.base, n_inst, total,
                               w.run_len, w.part_key, w.part_idx, t.flags, eidx, w.ovf, w.ovf_count, cap);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (n_seg > 0) {
        hipLaunchKernelGGL(table_segment_kernel, dim3((uint32_t)n_seg), dim3(kSegThreads), 0, s, t.keys, t.base,
                           t.nbuckets, seg_off, w.seg_inst, w.run_len, w.part_key, w.part_idx, w.ovf, w.ovf_count,
                           cap, entry_of, t.fp, t.fp_len, t.fp_inst);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(table_overflow_kernel, dim3((uint32_t)(4 * n_cu)), dim3(256), 0, s, t.keys, t.base,
                       t.nbuckets, inst_off, n_inst, hashes, total, w.part_key, w.ovf, w.ovf_count, cap, entry_of,
                       t.fp_extra,
                       t.fp_extra_inst, (uint32_t)(t.fp_extra_cap < 0xFFFFFFFFll ? t.fp_extra_cap : 0xFFFFFFFEll), t.fp_meta);
    return hipGetLastError();
}

}  // namespace ls
