// Prefix-index maintenance: commit a routed batch into the per-instance cache
// lists with exact least-recently-used eviction, then rebuild the tables.
//
// The gateway records each routed request's prefix blocks on the instance it
// chose, and each engine frees its least recently used KV blocks (Section 2;
// Section 4.2, Prefix KV cache tracker).  Every cached block carries a recency
// stamp (larger = more recent).  A commit of epoch e touches block k of routed
// request r with
//     e * 2^44 + r * 2^20 + (2^20 - 1 - k)
// (later commits, then later requests, then blocks nearer the prompt's start
// are more recent: an engine frees a sequence's tail first, so what stays of
// a request is a prefix of it); a block keeps its largest stamp.  Every
// instance above its capacity then keeps exactly its `capacity` most recent
// blocks.  Stamps are unique within an instance, so that set is exact.
//
// Device state beside the lookup tables: each instance's list of (hash,
// stamp) pairs (dense CSR), and for every table slot the list entry of the
// key in it (`entry_of`), so that a touch of a cached block raises that
// entry's stamp in place.  The all-ones key has no table slot; its entry is
// kept per instance (`eidx`).
//
// A commit, all on the stream:
//   occupancy   blocks routed to each instance (one atomic add per request)
//   layout      a batch-local hash set per instance for blocks not yet cached,
//               sized for its occupancy at half load
//   touch       one wave per request: cached -> atomic max on the entry's
//               stamp; not cached -> insert into the instance's set, atomic
//               max on the set slot's stamp
//   plan        candidates and survivors per instance, output offsets
//   select      one workgroup per instance: radix select (8 bits a pass, most
//               significant first) of the capacity-th largest stamp among the
//               candidates, then an order-preserving compaction of the
//               survivors into the new list
// followed by the table build on the new lists and a new entry map.
#include "ls_internal.h"

namespace ls {

constexpr int kStampKBits = 20, kStampRBits = 24;

__device__ __forceinline__ uint64_t commit_stamp(uint32_t epoch, uint32_t r, uint32_t k) {
    const uint32_t kmax = (1u << kStampKBits) - 1u;
    k = k < kmax ? k : kmax;                         // blocks past 2^20 - 1 share the last rank
    return ((uint64_t)epoch << (kStampKBits + kStampRBits)) | ((uint64_t)r << kStampKBits) | (uint64_t)(kmax - k);
}

// Slot (bucket * 8 + position) of `key` in a table of nb buckets, or -1.
// `key` must not be the all-ones key.
__device__ __forceinline__ int64_t find_slot(const uint64_t* __restrict__ table, uint32_t nb, uint64_t key) {
    uint32_t b = bucket_of(key, nb);
    for (uint32_t probe = 0; probe < nb; ++probe) {
        const ulonglong2* q = reinterpret_cast<const ulonglong2*>(table + (int64_t)b * kBucketKeys);
        const ulonglong2 v0 = q[0], v1 = q[1], v2 = q[2], v3 = q[3];
        const uint64_t slot[kBucketKeys] = {v0.x, v0.y, v1.x, v1.y, v2.x, v2.y, v3.x, v3.y};
#pragma unroll
        for (int s = 0; s < kBucketKeys; ++s) {
            if (slot[s] == key) return (int64_t)b * kBucketKeys + s;
            if (slot[s] == kEmptyKey) return -1;
        }
        b = (b + 1 == nb) ? 0 : b + 1;
    }
    return -1;
}

__device__ __forceinline__ int32_t owner_of_entry(const int64_t* __restrict__ off, int32_t n, int64_t t) {
    int32_t lo = 0, hi = n;                          // largest i with off[i] <= t
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (off[mid] <= t) lo = mid; else hi = mid;
    }
    return lo;
}

// Loaded lists: entry j of an instance gets stamp j + 1.
__global__ void position_stamps_kernel(const int64_t* __restrict__ off, int32_t N, uint64_t* __restrict__ stamp,
                                       int64_t total) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int32_t i = owner_of_entry(off, N, t);
        stamp[t] = (uint64_t)(t - off[i] + 1);
    }
}

// entry_of[slot of hash[j]] = the largest such j (the newest duplicate), and
// eidx[i] = the largest j holding the all-ones key.  Expects eidx = -1 and,
// where duplicates may exist, entry_of = 0 beforehand.
__global__ void entry_map_kernel(CacheTables T, const int64_t* __restrict__ off, int32_t N,
                                 const uint64_t* __restrict__ hash, uint32_t* __restrict__ entry_of,
                                 int64_t* __restrict__ eidx) {
    const int64_t total = off[N];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int32_t i = owner_of_entry(off, N, t);
        const uint64_t h = hash[t];
        if (h == kEmptyKey) {
            atomicMax((long long*)&eidx[i], (long long)t);   // eidx starts at -1: a signed max
            continue;
        }
        const int64_t base = T.base[i] * kBucketKeys;
        const int64_t q = find_slot(T.keys + base, T.nbuckets[i], h);
        if (q >= 0) atomicMax(&entry_of[base + q], (uint32_t)t);
    }
}

// Live flag of a loaded entry: the entry the map kept for its key.
__global__ void live_entries_kernel(CacheTables T, const int64_t* __restrict__ off, int32_t N,
                                    const uint64_t* __restrict__ hash, const uint32_t* __restrict__ entry_of,
                                    const int64_t* __restrict__ eidx, uint8_t* __restrict__ live) {
    const int64_t total = off[N];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int32_t i = owner_of_entry(off, N, t);
        const uint64_t h = hash[t];
        bool keep;
        if (h == kEmptyKey) {
            keep = eidx[i] == t;
        } else {
            const int64_t base = T.base[i] * kBucketKeys;
            const int64_t q = find_slot(T.keys + base, T.nbuckets[i], h);
            keep = q >= 0 && entry_of[base + q] == (uint32_t)t;
        }
        live[t] = keep ? 1 : 0;
    }
}

// Blocks routed to each instance: a workgroup sums its requests in LDS, then
// adds each non-zero count once (routing is often skewed to few instances).
constexpr int kOccLds = 8192;

__global__ __launch_bounds__(256) void occupancy_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                                        const int32_t* __restrict__ chosen, int32_t N,
                                                        int64_t* __restrict__ occ) {
    __shared__ unsigned long long part[kOccLds];
    const bool lds = N <= kOccLds;
    if (lds)
        for (int32_t i = threadIdx.x; i < N; i += blockDim.x) part[i] = 0;
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < R; r += stride) {
        const int32_t i = chosen[r];
        const int64_t n = req_off[r + 1] - req_off[r];
        if (i < 0 || i >= N || n <= 0) continue;
        if (lds) atomicAdd(&part[i], (unsigned long long)n);
        else atomicAdd((unsigned long long*)&occ[i], (unsigned long long)n);
    }
    __syncthreads();
    if (lds)
        for (int32_t i = threadIdx.x; i < N; i += blockDim.x)
            if (part[i]) atomicAdd((unsigned long long*)&occ[i], part[i]);
}

// Exclusive scan over N values in one workgroup of 1024 threads; out has N + 1
// entries.  value(i) is evaluated once per i.
template <typename F>
__device__ void block_scan_i64(int32_t N, F value, int64_t* __restrict__ out) {
    __shared__ int64_t part[1024];
    __shared__ int64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int32_t c0 = 0; c0 < N; c0 += 1024) {
        const int32_t i = c0 + (int32_t)threadIdx.x;
        const int64_t v = i < N ? value(i) : 0;
        part[threadIdx.x] = v;
        __syncthreads();
        for (int d = 1; d < 1024; d <<= 1) {           // inclusive Hillis-Steele scan
            const int64_t add = threadIdx.x >= (unsigned)d ? part[threadIdx.x - d] : 0;
            __syncthreads();
            part[threadIdx.x] += add;
            __syncthreads();
        }
        if (i < N) out[i] = carry + part[threadIdx.x] - v;
        __syncthreads();
        if (threadIdx.x == 1023) carry += part[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[N] = carry;
}

// Batch-local set layout: instance i gets max(1, ceil(occ_i / 4)) buckets.  If
// that exceeds the allocation (the caller's block count was too small), every
// set gets no bucket: blocks not yet cached are then dropped, nothing is
// written out of place.
__global__ __launch_bounds__(1024) void fresh_layout_kernel(int32_t N, const int64_t* __restrict__ occ,
                                                            int64_t cap_buckets, int64_t* __restrict__ fbase) {
    block_scan_i64(N, [&](int32_t i) -> int64_t { const int64_t b = (occ[i] + 3) / 4; return b < 1 ? 1 : b; },
                   fbase);
    __syncthreads();
    const bool over = fbase[N] > cap_buckets;
    __syncthreads();
    if (over)
        for (int32_t i = threadIdx.x; i <= N; i += blockDim.x) fbase[i] = 0;
}

// Empties the batch-local sets (the slot count is read on the device).
__global__ void fresh_clear_kernel(const int64_t* __restrict__ fbase, int32_t N, uint64_t* __restrict__ fkey,
                                   uint64_t* __restrict__ fstamp) {
    const int64_t total = fbase[N] * kBucketKeys;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        fkey[t] = kEmptyKey;
        fstamp[t] = 0;
    }
}

// Reads of words other waves update with atomics: device-scope loads, which
// see those updates rather than a stale line of this CU's cache.
__device__ __forceinline__ uint64_t load_shared(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// *p = max(*p, s).  Stamps only grow, so a read can only be smaller than the
// current value: the atomic is skipped only when it could not change *p.
__device__ __forceinline__ void raise_stamp(uint64_t* p, uint64_t s) {
    if (load_shared(p) < s) atomicMax((unsigned long long*)p, (unsigned long long)s);
}

// One wave per request: touch each of its blocks on the chosen instance.
constexpr int kTouchWaves = 4;

__global__ __launch_bounds__(kTouchWaves * 64) void touch_kernel(
    CacheTables T, int32_t R, const int64_t* __restrict__ req_off, const uint64_t* __restrict__ req_hashes,
    const int32_t* __restrict__ chosen, int32_t N, uint32_t epoch, const uint32_t* __restrict__ entry_of,
    const int64_t* __restrict__ eidx, uint64_t* __restrict__ stamp, const int64_t* __restrict__ fbase,
    uint64_t* __restrict__ fkey, uint64_t* __restrict__ fstamp, int64_t* __restrict__ fcount,
    uint64_t* __restrict__ efresh) {
    const int lane = threadIdx.x & 63;
    const int64_t wstride = (int64_t)gridDim.x * kTouchWaves;
    // Later requests carry larger stamps, so they go first: a block shared by
    // many requests then mostly sees its final stamp already there, and the
    // read below skips the atomic.
    for (int64_t rr = (int64_t)blockIdx.x * kTouchWaves + (threadIdx.x >> 6); rr < R; rr += wstride) {
        const int64_t r = R - 1 - rr;
        const int32_t i = chosen[r];
        if (i < 0 || i >= N) continue;
        const int64_t o = req_off[r], n = req_off[r + 1] - o;
        const int64_t tbase = T.base[i] * kBucketKeys;
        const uint32_t tnb = T.nbuckets[i];
        const int64_t fb = fbase[i];
        const uint32_t fnb = (uint32_t)(fbase[i + 1] - fb);
        uint64_t* fk = fkey + fb * kBucketKeys;
        uint64_t* fs = fstamp + fb * kBucketKeys;
        uint32_t claimed = 0;                            // set slots this lane filled
        for (int64_t k = lane; k < n; k += 64) {
            const uint64_t h = req_hashes[o + k];
            const uint64_t s = commit_stamp(epoch, (uint32_t)r, (uint32_t)k);
            if (h == kEmptyKey) {
                const int64_t e = eidx[i];
                raise_stamp(e >= 0 ? &stamp[e] : &efresh[i], s);
                continue;
            }
            const int64_t q = find_slot(T.keys + tbase, tnb, h);
            if (q >= 0) {
                raise_stamp(&stamp[entry_of[tbase + q]], s);
                continue;
            }
            // not cached: into the instance's batch-local set (a slot changes at
            // most once, empty -> key; the set never fills: it is at most half full)
            uint32_t b = bucket_of(h, fnb);
            for (uint32_t probe = 0; probe < fnb; ++probe) {
                int64_t at = -1;
                for (int sl = 0; sl < kBucketKeys; ++sl) {
                    const int64_t slot = (int64_t)b * kBucketKeys + sl;
                    uint64_t cur = load_shared(&fk[slot]);
                    if (cur == kEmptyKey) {
                        cur = atomicCAS((unsigned long long*)&fk[slot], (unsigned long long)kEmptyKey,
                                        (unsigned long long)h);
                        if (cur == kEmptyKey) {
                            ++claimed;
                            at = slot;
                            break;
                        }
                    }
                    if (cur == h) {
                        at = slot;
                        break;
                    }
                }
                if (at >= 0) {
                    raise_stamp(&fs[at], s);
                    break;
                }
                b = (b + 1 == fnb) ? 0 : b + 1;
            }
        }
        // one count per request (the wave's lanes all serve this instance)
        for (int d = 32; d > 0; d >>= 1) claimed += __shfl_xor(claimed, d);
        if (lane == 0 && claimed) atomicAdd((unsigned long long*)&fcount[i], (unsigned long long)claimed);
    }
}

// Live entries per instance (one workgroup each), then their offsets.
__global__ __launch_bounds__(1024) void count_live_kernel(const int64_t* __restrict__ off,
                                                          const uint8_t* __restrict__ live, int64_t* __restrict__ cand) {
    __shared__ int64_t part[1024];
    const int32_t i = blockIdx.x;
    int64_t n = 0;
    for (int64_t t = off[i] + threadIdx.x; t < off[i + 1]; t += 1024) n += live[t];
    part[threadIdx.x] = n;
    __syncthreads();
    for (int d = 512; d > 0; d >>= 1) {
        if (threadIdx.x < (unsigned)d) part[threadIdx.x] += part[threadIdx.x + d];
        __syncthreads();
    }
    if (threadIdx.x == 0) cand[i] = part[0];
}

__global__ __launch_bounds__(1024) void scan_counts_kernel(int32_t N, const int64_t* __restrict__ cand,
                                                           int64_t* __restrict__ off2) {
    block_scan_i64(N, [&](int32_t i) -> int64_t { return cand[i]; }, off2);
}

// Candidates t_i = listed + fresh, survivors min(t_i, capacity_i), output
// offsets; candidate chunks per instance for the selection passes; the
// selection state (an instance selects only if t_i > capacity_i).
__global__ __launch_bounds__(1024) void commit_plan_kernel(IndexCommit C) {
    const int32_t N = C.N;
    for (int32_t i = threadIdx.x; i < N; i += blockDim.x) {
        const int64_t nold = C.off[i + 1] - C.off[i];
        const int64_t nf = (C.fbase[i + 1] - C.fbase[i]) * kBucketKeys;
        C.cand[i] = nold + C.fcount[i] + (C.efresh[i] != 0 ? 1 : 0);
        C.nvirt[i] = nold + nf + 1;                      // listed entries, set slots, the all-ones key
        const int64_t keep = C.cand[i] < C.capacity[i] ? C.cand[i] : C.capacity[i];
        C.sel_want[i] = keep;
        C.sel_prefix[i] = 0;
        C.sel_mask[i] = 0;
        C.sel_pos[i] = 0;
        C.sel_active[i] = C.cand[i] > keep ? 1 : 0;
    }
    __syncthreads();
    block_scan_i64(N, [&](int32_t i) -> int64_t { return C.cand[i] < C.capacity[i] ? C.cand[i] : C.capacity[i]; },
                   C.off2);
    __syncthreads();
    block_scan_i64(N, [&](int32_t i) -> int64_t { return (C.nvirt[i] + kSelChunk - 1) / kSelChunk; }, C.chunk0);
    for (int64_t t = threadIdx.x; t < (int64_t)N * 256; t += blockDim.x) C.sel_hist[t] = 0;
}

// The candidates of one instance: listed entries, set slots, the fresh
// all-ones key (position nold + nf).  Read once per chunk.
struct CandView {
    const uint64_t* hash;
    const uint64_t* stamp;
    const uint64_t* fk;
    const uint64_t* fs;
    int64_t nold, nf;
    uint64_t ef;
    __device__ __forceinline__ bool get(int64_t v, uint64_t& h, uint64_t& s) const {
        if (v < nold) {
            h = hash[v];
            s = stamp[v];
            return true;
        }
        if (v < nold + nf) {
            h = fk[v - nold];
            s = fs[v - nold];
            return h != kEmptyKey;
        }
        h = kEmptyKey;
        s = ef;
        return ef != 0;
    }
};

__device__ __forceinline__ CandView cand_view(const IndexCommit& C, int32_t i) {
    CandView V;
    const int64_t o0 = C.off[i];
    V.nold = C.off[i + 1] - o0;
    V.hash = C.hash + o0;
    V.stamp = C.stamp + o0;
    const int64_t f0 = C.fbase[i] * kBucketKeys;
    V.nf = (C.fbase[i + 1] - C.fbase[i]) * kBucketKeys;
    V.fk = C.fkey + f0;
    V.fs = C.fstamp + f0;
    V.ef = C.efresh[i];
    return V;
}

// One selection pass (digit `shift / 8`): histogram of the digit over each
// selecting instance's candidates that match its prefix so far.
__global__ __launch_bounds__(256) void select_hist_kernel(IndexCommit C, int shift) {
    __shared__ uint32_t lh[256];
    const int64_t nchunks = C.chunk0[C.N];
    for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const int32_t i = owner_of_entry(C.chunk0, C.N, ch);
        if (!C.sel_active[i]) continue;                  // uniform over the workgroup
        lh[threadIdx.x] = 0;
        __syncthreads();
        const uint64_t prefix = C.sel_prefix[i], mask = C.sel_mask[i];
        const CandView V = cand_view(C, i);
        const int64_t v0 = (ch - C.chunk0[i]) * kSelChunk;
        const int64_t v1 = v0 + kSelChunk < C.nvirt[i] ? v0 + kSelChunk : C.nvirt[i];
        // all of the thread's candidates are loaded before any is used, so the
        // loads are in flight together
        constexpr int kPer = (int)(kSelChunk / 256);
        uint64_t st[kPer];
        bool ok[kPer];
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int64_t v = v0 + threadIdx.x + (int64_t)u * 256;
            uint64_t h;
            ok[u] = v < v1 && V.get(v, h, st[u]);
        }
#pragma unroll
        for (int u = 0; u < kPer; ++u)
            if (ok[u] && (st[u] & mask) == prefix) atomicAdd(&lh[(st[u] >> shift) & 255u], 1u);
        __syncthreads();
        if (lh[threadIdx.x]) atomicAdd(&C.sel_hist[(int64_t)i * 256 + threadIdx.x], lh[threadIdx.x]);
        __syncthreads();
    }
}

// The digit of the want-th largest candidate: the highest bin d >= 1 whose
// count, added to the counts of the bins above it, reaches `want` (bin 0 when
// none does).  One wave per instance: lane l holds bins 255 - 4l .. 252 - 4l,
// and a scan across the lanes gives each the counts above its bins.  The
// histogram is cleared for the next pass.
__global__ __launch_bounds__(256) void select_digit_kernel(IndexCommit C, int shift) {
    const int32_t i = (int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (i >= C.N || !C.sel_active[i]) return;           // uniform over the wave
    uint32_t* hh = C.sel_hist + (int64_t)i * 256;
    uint32_t cnt[4];
    int64_t mine = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        cnt[q] = hh[255 - 4 * lane - q];
        mine += cnt[q];
    }
    int64_t incl = mine;
#pragma unroll
    for (int dd = 1; dd < 64; dd <<= 1) {
        const int64_t t = __shfl_up(incl, dd);
        if (lane >= dd) incl += t;
    }
    const int64_t want = C.sel_want[i];
    int64_t cum = incl - mine, cum_at = 0;
    int found = -1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int bin = 255 - 4 * lane - q;
        if (found < 0 && bin >= 1 && cum + (int64_t)cnt[q] >= want) {
            found = bin;
            cum_at = cum;
        }
        cum += cnt[q];
    }
    const uint64_t m = __ballot(found >= 0);
    int digit;
    int64_t above;
    if (m) {
        const int first = __ffsll((long long)m) - 1;
        digit = __shfl(found, first);
        above = __shfl(cum_at, first);
    } else {
        digit = 0;                                       // every bin but 0: the total less bin 0 (lane 63)
        above = __shfl(incl, 63) - (int64_t)__shfl((int)cnt[3], 63);
    }
    if (lane == 0) {
        C.sel_want[i] = want - above;
        C.sel_prefix[i] |= (uint64_t)digit << shift;
        C.sel_mask[i] |= 255ull << shift;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) hh[255 - 4 * lane - q] = 0;
}

// Survivors (stamp >= the selected one, or all) into the new lists: a chunk
// (never spanning two instances) counts its survivors, takes its place with one
// atomic add, and writes them at offsets from a workgroup scan (thread t takes
// candidates t, t + 256, ... of the chunk, so reads stay coalesced).
__global__ __launch_bounds__(256) void select_compact_multi_kernel(IndexCommit C) {
    constexpr int kPer = (int)(kSelChunk / 256);      // candidates per thread and chunk, strided by 256
    __shared__ uint32_t wsum[4];
    __shared__ int64_t s_base;
    const int64_t nchunks = C.chunk0[C.N];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const int32_t i = owner_of_entry(C.chunk0, C.N, ch);
        const uint64_t theta = C.sel_active[i] ? C.sel_prefix[i] : 0;
        const int64_t keep = C.off2[i + 1] - C.off2[i];
        const int64_t v0 = (ch - C.chunk0[i]) * kSelChunk + threadIdx.x;
        const int64_t vend = C.nvirt[i];
        const CandView V = cand_view(C, i);
        uint64_t* dh = C.hash2 + C.off2[i];
        uint64_t* ds = C.stamp2 + C.off2[i];
        // the thread's candidates, read once and all in flight together
        uint64_t hh[kPer], ss[kPer];
        bool kept[kPer];
        uint32_t mine = 0;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int64_t v = v0 + (int64_t)u * 256;
            kept[u] = v < vend && V.get(v, hh[u], ss[u]);
        }
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            kept[u] = kept[u] && ss[u] >= theta;
            mine += kept[u] ? 1u : 0u;
        }
        // exclusive scan of `mine` over the workgroup (in thread order)
        uint32_t incl = mine;
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t t = __shfl_up(incl, d);
            if (lane >= d) incl += t;
        }
        if (lane == 63) wsum[wv] = incl;
        __syncthreads();
        uint32_t before = incl - mine;
        for (int w = 0; w < wv; ++w) before += wsum[w];
        if (threadIdx.x == 0) {
            const uint32_t tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
            s_base = tot ? (int64_t)atomicAdd((unsigned long long*)&C.sel_pos[i], (unsigned long long)tot) : 0;
        }
        __syncthreads();
        int64_t pos = s_base + before;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            if (kept[u]) {
                if (pos < keep) {
                    dh[pos] = hh[u];
                    ds[pos] = ss[u];
                }
                ++pos;
            }
        }
        __syncthreads();
    }
}

// Loaded lists without repeated keys: one workgroup per instance keeps its
// live entries, in list order (a workgroup scan per chunk of 1024 entries).
constexpr int kSelThreads = 1024;

struct SelectArgs {
    const int64_t* off;           // current lists
    const uint64_t* hash;
    const uint64_t* stamp;
    const uint8_t* live;
    const int64_t* off2;          // new lists
    uint64_t* hash2;
    uint64_t* stamp2;
};

__global__ __launch_bounds__(kSelThreads) void select_compact_kernel(SelectArgs A) {
    __shared__ uint32_t wcount[kSelThreads / 64];
    __shared__ int64_t s_base;
    const int32_t i = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t o0 = A.off[i], n = A.off[i + 1] - o0;
    const int64_t keep = A.off2[i + 1] - A.off2[i];
    if (tid == 0) s_base = 0;
    __syncthreads();
    uint64_t* dh = A.hash2 + A.off2[i];
    uint64_t* ds = A.stamp2 + A.off2[i];
    for (int64_t c0 = 0; c0 < n; c0 += kSelThreads) {
        const int64_t idx = c0 + tid;
        const bool in = idx < n && A.live[o0 + idx] != 0;
        const uint64_t m = __ballot(in);
        if (lane == 0) wcount[wv] = (uint32_t)__popcll(m);
        __syncthreads();
        int64_t before = s_base;
        for (int w = 0; w < wv; ++w) before += wcount[w];
        before += __popcll(m & ((1ull << lane) - 1ull));
        if (in && before < keep) {
            dh[before] = A.hash[o0 + idx];
            ds[before] = A.stamp[o0 + idx];
        }
        __syncthreads();
        if (tid == 0) {
            int64_t tot = 0;
            for (int w = 0; w < kSelThreads / 64; ++w) tot += wcount[w];
            s_base += tot;
        }
        __syncthreads();
    }
}

static int grid_of(int64_t n, int block, int n_cu) {
    int64_t g = (n + block - 1) / block;
    const int64_t cap = (int64_t)n_cu * 16;
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (int)g;
}

hipError_t launch_position_stamps(const int64_t* off, int32_t N, uint64_t* stamp, int64_t total, int n_cu,
                                  hipStream_t s) {
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(position_stamps_kernel, dim3(grid_of(total, 256, n_cu)), dim3(256), 0, s, off, N, stamp,
                       total);
    return hipGetLastError();
}

hipError_t launch_entry_map(const CacheTables& T, const int64_t* off, int32_t N, const uint64_t* hash,
                            uint32_t* entry_of, int64_t* eidx, int64_t total_bound, int n_cu, hipStream_t s) {
    hipError_t e = launch_fill_u64(reinterpret_cast<uint64_t*>(eidx), ~0ull, N, s);
    if (e != hipSuccess) return e;
    if (total_bound <= 0) return hipSuccess;
    hipLaunchKernelGGL(entry_map_kernel, dim3(grid_of(total_bound, 256, n_cu)), dim3(256), 0, s, T, off, N, hash,
                       entry_of, eidx);
    return hipGetLastError();
}

hipError_t launch_live_entries(const CacheTables& T, const int64_t* off, int32_t N, const uint64_t* hash,
                               const uint32_t* entry_of, const int64_t* eidx, uint8_t* live, int64_t total_bound,
                               int n_cu, hipStream_t s) {
    if (total_bound <= 0) return hipSuccess;
    hipLaunchKernelGGL(live_entries_kernel, dim3(grid_of(total_bound, 256, n_cu)), dim3(256), 0, s, T, off, N, hash,
                       entry_of, eidx, live);
    return hipGetLastError();
}

// Loaded lists without duplicate keys: the newest of each, in list order.
hipError_t launch_dedup_lists(const int64_t* off, int32_t N, const uint64_t* hash, const uint64_t* stamp,
                              const uint8_t* live, int64_t* cand, int64_t* off2, uint64_t* hash2, uint64_t* stamp2,
                              hipStream_t s) {
    // cand_i = live entries; off2 = their scan (no capacity)
    hipLaunchKernelGGL(count_live_kernel, dim3((uint32_t)N), dim3(1024), 0, s, off, live, cand);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(1024), 0, s, N, cand, off2);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SelectArgs A{};
    A.off = off; A.hash = hash; A.stamp = stamp; A.live = live;
    A.off2 = off2; A.hash2 = hash2; A.stamp2 = stamp2;
    hipLaunchKernelGGL(select_compact_kernel, dim3((uint32_t)N), dim3(kSelThreads), 0, s, A);
    return hipGetLastError();
}

hipError_t launch_commit(const CacheTables& T, const IndexCommit& C, hipStream_t s) {
    const int32_t N = C.N;
    hipError_t e;
    const FillOp fills[3] = {{C.occ, 0u, N, 8}, {C.fcount, 0u, N, 8}, {C.efresh, 0u, N, 8}};
    if ((e = launch_fill_multi(fills, 3, s)) != hipSuccess) return e;
    if (C.R > 0) {
        hipLaunchKernelGGL(occupancy_kernel, dim3(grid_of(C.R, 256, C.n_cu)), dim3(256), 0, s, C.R, C.req_off,
                           C.chosen, N, C.occ);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fresh_layout_kernel, dim3(1), dim3(1024), 0, s, N, C.occ,
                       C.fresh_slots_bound / kBucketKeys, C.fbase);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(fresh_clear_kernel, dim3(grid_of(C.fresh_slots_bound, 256, C.n_cu)), dim3(256), 0, s, C.fbase,
                       N, C.fkey, C.fstamp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (C.R > 0) {
        int64_t g = ((int64_t)C.R + kTouchWaves - 1) / kTouchWaves;
        if (g > (int64_t)C.n_cu * 16) g = (int64_t)C.n_cu * 16;
        hipLaunchKernelGGL(touch_kernel, dim3((uint32_t)g), dim3(kTouchWaves * 64), 0, s, T, C.R, C.req_off,
                           C.req_hashes, C.chosen, N, C.epoch, C.entry_of, C.eidx, C.stamp, C.fbase, C.fkey,
                           C.fstamp, C.fcount, C.efresh);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(commit_plan_kernel, dim3(1), dim3(1024), 0, s, C);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int grid = grid_of(C.chunk_bound * 256, 256, C.n_cu);
    for (int p = 7; p >= 0; --p) {
        hipLaunchKernelGGL(select_hist_kernel, dim3(grid), dim3(256), 0, s, C, 8 * p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(select_digit_kernel, dim3((uint32_t)((N + 3) / 4)), dim3(256), 0, s, C, 8 * p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_compact_multi_kernel, dim3(grid), dim3(256), 0, s, C);
    return hipGetLastError();
}

}  // namespace ls
