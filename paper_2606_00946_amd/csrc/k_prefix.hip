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
// Continuations.  Where l[lead,i] >= c, the follower's run goes on from block
// c, whose hash is usually the follower's own (its question after a shared
// template) and cached nowhere.  For a large batch the library first collects
// those continuation hashes in a small table and marks, in one sequential pass
// over every cached key, the ones some instance holds (a semi-join).  A
// follower whose continuation is cached nowhere has l[r,i] = c wherever
// l[lead,i] >= c, with no probe; only the others are probed.
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
constexpr int32_t kContNone = -1;    // follower's prompt ends within the common prefix
constexpr int32_t kContProbe = -2;   // continuation must be probed

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

// The same run with a whole wave on one pair: group g of four lanes probes
// blocks l + g + 16 t (t < TS), so one round covers up to 16 TS positions.  The
// window starts at W and doubles after every all-hit round (..., 16 TS): long
// runs advance 16 TS blocks per dependent round, short ones waste little.  (A
// window of 256 positions, TS = 16, was slower on 5,000-block runs over
// 400,000-key tables: the random bucket reads, not the rounds, bound it.)
template <int TS = 4>
__device__ __forceinline__ int64_t extend_run_wave(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                                   const uint64_t* __restrict__ h, int64_t n, int64_t l, int lane,
                                                   int W = 4) {
    constexpr int WMAX = 16 * TS;
    const int g = lane >> 2, q = lane & 3, shift = g * 4;
    // the window's block hashes; the next window's are read while this one's
    // buckets are in flight (used only if every probe of this window hits)
    uint64_t key[TS];
    bool act[TS];
    auto load_keys = [&](int64_t l0, int w, uint64_t (&k)[TS], bool (&a)[TS]) {
#pragma unroll
        for (int t = 0; t < TS; ++t) {
            a[t] = g + 16 * t < w && l0 + g + 16 * t < n;
            if (a[t]) k[t] = h[l0 + g + 16 * t];
        }
    };
    load_keys(l, W, key, act);
    while (l < n) {
        ulonglong2 v[TS];
        uint32_t bkt[TS];
#pragma unroll
        for (int t = 0; t < TS; ++t) {
            if (act[t]) {
                bkt[t] = bucket_of(key[t], nb);
                v[t] = *reinterpret_cast<const ulonglong2*>(table + (int64_t)bkt[t] * kBucketKeys + q * 2);
            }
        }
        const int64_t ln = l + W < n ? l + W : n;
        const int Wn = W * 2 > WMAX ? WMAX : W * 2;
        uint64_t nkey[TS];
        bool nact[TS];
        load_keys(ln, Wn, nkey, nact);
        int64_t stop = -1;
#pragma unroll
        for (int t = 0; t < TS; ++t) {
            if (16 * t >= W || stop >= 0) break;            // uniform across the wave
            bool hit = true;
            if (act[t]) {
                if (key[t] == kEmptyKey) {
                    hit = has_empty;
                } else {
                    const uint64_t kk = key[t];
                    bool found = (v[t].x == kk) | (v[t].y == kk);
                    bool empty = (v[t].x == kEmptyKey) | (v[t].y == kEmptyKey);
                    bool gfound = ((__ballot(found) >> shift) & 0xFull) != 0;
                    bool gempty = ((__ballot(empty) >> shift) & 0xFull) != 0;
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
            }
            const uint64_t miss = __ballot(q == 0 && act[t] && !hit);
            if (miss) stop = l + 16 * t + ((__ffsll((long long)miss) - 1) >> 2);
        }
        if (stop >= 0) return stop;
        l = ln;
        W = Wn;
#pragma unroll
        for (int t = 0; t < TS; ++t) {
            key[t] = nkey[t];
            act[t] = nact[t];
        }
    }
    return l;
}

// Prefix-closed caches.  When every instance's cached set is prefix-closed for
// every prompt (if block j of a prompt is cached, so are its blocks 0..j-1 --
// the state an engine's tail-first LRU keeps), whether block j is cached is a
// non-increasing function of j and the run is its first miss.  A wave then
// searches instead of walking: each round probes 16 positions spread over the
// open interval [lo, hi) (group g takes lo + (g + 1)(hi - lo) / 17, or lo + g
// when the interval is short), which shrinks it about 17-fold; about four
// rounds settle an 8k-block prompt.  Exact only under that invariant.
__device__ __forceinline__ bool probe_block(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                           uint64_t key, int q, int shift) {
    if (key == kEmptyKey) return has_empty;
    uint32_t b = bucket_of(key, nb);
    for (uint32_t probe = 0; probe < nb; ++probe) {
        const ulonglong2 w = *reinterpret_cast<const ulonglong2*>(table + (int64_t)b * kBucketKeys + q * 2);
        const bool found = (w.x == key) | (w.y == key);
        const bool empty = (w.x == kEmptyKey) | (w.y == kEmptyKey);
        if (((__ballot(found) >> shift) & 0xFull) != 0) return true;
        if (((__ballot(empty) >> shift) & 0xFull) != 0) return false;
        b = (b + 1 == nb) ? 0 : b + 1;
    }
    return false;
}

__device__ __forceinline__ int64_t search_run_wave(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                                   const uint64_t* __restrict__ h, int64_t n, int lane) {
    const int g = lane >> 2, q = lane & 3, shift = g * 4;
    int64_t lo = 0, hi = n;                      // blocks [0, lo) cached; block hi is the first miss (or n)
    while (lo < hi) {
        const int64_t lo0 = lo, span = hi - lo;
        // probed positions, increasing with the group index; all inside [lo0, hi)
        auto pos = [&](int gg) -> int64_t { return span > 16 ? lo0 + ((int64_t)(gg + 1) * span) / 17 : lo0 + gg; };
        const int64_t j = pos(g);
        const bool act = j < hi;
        bool hit = false;
        if (act) hit = probe_block(table, nb, has_empty, h[j], q, shift);
        const uint64_t hits = __ballot(q == 0 && act && hit);
        const uint64_t miss = __ballot(q == 0 && act && !hit);
        if (hits) lo = pos((63 - __clzll((long long)hits)) >> 2) + 1;
        if (miss) hi = pos((__ffsll((long long)miss) - 1) >> 2);
    }
    return lo;
}

// ---------------------------------------------------------------------------
// grouping by first block hash
// ---------------------------------------------------------------------------
// slot of request r in the group table (-1: ungrouped, r leads itself); the
// group's leader word keeps max over members of (n_r << 32 | ~r): longest
// prompt, lowest id on ties.
// A workgroup first collects its members' first hashes in an LDS table and
// combines their words there; one thread per distinct hash then inserts it in
// the global table and raises the group's word.  A popular group therefore
// costs one global compare-and-swap and one atomic per workgroup, not per
// member.
constexpr int kGroupThreads = 1024;
constexpr int kGroupLds = 2048;      // LDS table entries (>= 2 x threads)

__global__ __launch_bounds__(kGroupThreads) void group_insert_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                                                     const uint64_t* __restrict__ req_hashes,
                                                                     uint64_t* __restrict__ gkeys,
                                                                     unsigned long long* __restrict__ glead,
                                                                     uint32_t G, int32_t* __restrict__ slot_of) {
    __shared__ uint64_t lkey[kGroupLds];
    __shared__ unsigned long long lword[kGroupLds];
    __shared__ int32_t lslot[kGroupLds];
    for (int e = threadIdx.x; e < kGroupLds; e += kGroupThreads) {
        lkey[e] = kEmptyKey;
        lword[e] = 0ull;
        lslot[e] = -1;
    }
    __syncthreads();
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t n = r < R ? req_off[r + 1] - req_off[r] : 0;
    int lidx = -1;
    if (n > 0) {
        const uint64_t key = req_hashes[req_off[r]];
        if (key != kEmptyKey) {
            uint32_t h = bucket_of(key, kGroupLds);
            for (int probe = 0; probe < kGroupLds; ++probe) {
                const unsigned long long old = atomicCAS((unsigned long long*)&lkey[h], (unsigned long long)kEmptyKey,
                                                         (unsigned long long)key);
                if (old == kEmptyKey || old == key) {
                    lidx = (int)h;
                    break;
                }
                h = (h + 1 == (uint32_t)kGroupLds) ? 0 : h + 1;
            }
            const unsigned long long word =
                ((unsigned long long)n << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)r);
            if (lidx >= 0) atomicMax(&lword[lidx], word);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kGroupLds; e += kGroupThreads) {
        const uint64_t key = lkey[e];
        if (key == kEmptyKey) continue;
        int32_t slot = -1;
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
        lslot[e] = slot;
        if (slot >= 0 && glead[slot] < lword[e]) atomicMax(glead + slot, lword[e]);
    }
    __syncthreads();
    if (r < R) slot_of[r] = lidx >= 0 ? lslot[lidx] : -1;
}

// Continuation table: open addressing over G slots of uint64 keys.
__device__ __forceinline__ int32_t cont_insert(uint64_t* __restrict__ qkeys, uint32_t G, uint64_t key) {
    uint32_t b = bucket_of(key, G);
    for (uint32_t probe = 0; probe < G; ++probe) {
        const uint64_t cur = qkeys[b];
        if (cur == key) return (int32_t)b;
        if (cur == kEmptyKey) {
            const unsigned long long old = atomicCAS((unsigned long long*)(qkeys + b), (unsigned long long)kEmptyKey,
                                                     (unsigned long long)key);
            if (old == kEmptyKey || old == key) return (int32_t)b;
        }
        b = (b + 1 == G) ? 0 : b + 1;
    }
    return kContProbe;
}

// One wave per request: leader id and common-prefix length with the leader;
// leaders append themselves to the leader list.  With the semi-join on, a
// follower registers the hash of its block c (cont_of: slot, kContNone when c
// reaches its end, kContProbe when it must be probed).
__global__ __launch_bounds__(256) void group_lcp_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                                        const uint64_t* __restrict__ req_hashes,
                                                        const unsigned long long* __restrict__ glead,
                                                        const int32_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ lead_of, int32_t* __restrict__ lcp_of,
                                                        int32_t* __restrict__ leaders, uint32_t* __restrict__ n_leaders,
                                                        uint64_t* __restrict__ qkeys, uint32_t G,
                                                        int32_t* __restrict__ cont_of, int join) {
    // 16 lanes per request (four requests per wave): the chain of dependent
    // reads before the compare is the cost, so more requests in flight pay.  A
    // round compares 16 w positions, lane sl taking j0 + sl + 16 u (u < w), all
    // loads issued before any compare; w doubles after every all-equal round
    // (1, 2, 4, 8), so long common prefixes take few dependent rounds.
    constexpr int kLcpMaxLoads = 8;
    const int lane = threadIdx.x & 63, sg = lane >> 4, sl = lane & 15;
    const int64_t r = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 4 + sg;
    if (r >= R) return;                               // uniform over the 16 lanes
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
        int w = 1;
        for (int64_t j0 = 0; j0 < m; j0 += 16 * w, w = w * 2 > kLcpMaxLoads ? kLcpMaxLoads : w * 2) {
            uint64_t av[kLcpMaxLoads], bv[kLcpMaxLoads];
#pragma unroll
            for (int u = 0; u < kLcpMaxLoads; ++u) {
                const int64_t j = j0 + sl + 16 * u;
                if (u < w && j < m) {
                    av[u] = a[j];
                    bv[u] = b[j];
                }
            }
            int64_t first = m;                       // this lane's first differing position
#pragma unroll
            for (int u = kLcpMaxLoads - 1; u >= 0; --u) {
                const int64_t j = j0 + sl + 16 * u;
                if (u < w && j < m && av[u] != bv[u]) first = j;
            }
#pragma unroll
            for (int off = 8; off >= 1; off >>= 1) {
                const int64_t o = __shfl_xor(first, off, 16);
                first = o < first ? o : first;
            }
            if (first < m) {                          // uniform over the 16 lanes
                c = first;
                break;
            }
        }
    }
    if (sl == 0) {
        lead_of[r] = (int32_t)lead;
        lcp_of[r] = (int32_t)c;
        if (lead == r) leaders[atomicAdd(n_leaders, 1u)] = (int32_t)r;
        int32_t cont = kContNone;
        if (lead != r && c < n) {
            const uint64_t key = req_hashes[req_off[r] + c];
            cont = (join && key != kEmptyKey) ? cont_insert(qkeys, G, key) : kContProbe;
        }
        cont_of[r] = cont;
    }
}

// The semi-join pass: every cached key looks itself up among the continuation
// hashes and marks the ones it finds.  A two-bit Bloom filter of the
// continuation hashes (kContFilterBits) sits in LDS, so the scan streams the
// tables and tests two LDS bits per key; keys that pass go on a list, and a
// second kernel looks them up in the continuation table.  If the list
// overflows, every continuation is marked seen (its followers are probed, so
// the overlaps stay exact).
constexpr int kContFilterLog = 20;
constexpr int kContFilterWords = (1 << kContFilterLog) / 32;     // 128 KiB
constexpr int kContThreads = 1024;
constexpr int64_t kContListCap = 1 << 22;

__device__ __forceinline__ void cont_bits(uint64_t key, uint32_t& b0, uint32_t& b1) {
    const uint64_t x = key * 0xD6E8FEB86659FD93ull;
    b0 = (uint32_t)(x >> (64 - kContFilterLog));
    b1 = (uint32_t)(x >> 8) & ((1u << kContFilterLog) - 1);
}

__global__ void cont_filter_kernel(const uint64_t* __restrict__ qkeys, uint32_t G, uint32_t* __restrict__ filter) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= G) return;
    const uint64_t key = qkeys[b];
    if (key == kEmptyKey) return;
    uint32_t b0, b1;
    cont_bits(key, b0, b1);
    atomicOr(&filter[b0 >> 5], 1u << (b0 & 31));
    atomicOr(&filter[b1 >> 5], 1u << (b1 & 31));
}

// Workgroup b appends the keys that pass the filter to its own slice of the
// candidate list (cap entries, counted in LDS); no global counter is shared.
__global__ __launch_bounds__(kContThreads) void cont_scan_kernel(const uint64_t* __restrict__ keys, int64_t n_slots,
                                                                 const uint32_t* __restrict__ filter,
                                                                 uint64_t* __restrict__ cand, uint32_t cap,
                                                                 uint32_t* __restrict__ n_cand) {
    __shared__ uint32_t lf[kContFilterWords];
    __shared__ uint32_t lcount;
    {
        const uint4* __restrict__ f4 = reinterpret_cast<const uint4*>(filter);
        uint4* l4 = reinterpret_cast<uint4*>(lf);
        for (int e = threadIdx.x; e < kContFilterWords / 4; e += kContThreads) l4[e] = f4[e];
        if (threadIdx.x == 0) lcount = 0u;
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    uint64_t* __restrict__ mine = cand + (int64_t)blockIdx.x * cap;
    const ulonglong2* __restrict__ k2 = reinterpret_cast<const ulonglong2*>(keys);
    const int64_t n2 = n_slots / 2;
    const int64_t stride = (int64_t)gridDim.x * kContThreads;
    // every lane runs the same number of iterations (the ballots below need the whole wave)
    for (int64_t e0 = (int64_t)blockIdx.x * kContThreads + threadIdx.x; e0 - threadIdx.x < n2; e0 += 4 * stride) {
        ulonglong2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t e = e0 + u * stride;
            v[u] = e < n2 ? k2[e] : ulonglong2{kEmptyKey, kEmptyKey};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint64_t kk[2] = {v[u].x, v[u].y};
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const uint64_t key = kk[j];
                bool pass = false;
                if (key != kEmptyKey) {
                    uint32_t b0, b1;
                    cont_bits(key, b0, b1);
                    pass = ((lf[b0 >> 5] >> (b0 & 31)) & 1u) && ((lf[b1 >> 5] >> (b1 & 31)) & 1u);
                }
                const uint64_t m = __ballot(pass);
                if (m) {
                    const int first = __ffsll((long long)m) - 1;
                    uint32_t base = 0;
                    if (lane == first) base = atomicAdd(&lcount, (uint32_t)__popcll(m));
                    base = (uint32_t)__shfl((int)base, first);
                    const uint32_t pos = base + (uint32_t)__popcll(m & ((1ull << lane) - 1));
                    if (pass && pos < cap) mine[pos] = key;
                }
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) n_cand[blockIdx.x] = lcount;
}

// Block b looks up slice b.  A slice that overflowed marks every continuation
// seen (its keys are lost, so their followers must be probed).
__global__ __launch_bounds__(256) void cont_probe_kernel(const uint64_t* __restrict__ cand, uint32_t cap,
                                                         const uint32_t* __restrict__ n_cand,
                                                         const uint64_t* __restrict__ qkeys, uint32_t G,
                                                         uint32_t* __restrict__ qseen) {
    const uint32_t cnt = n_cand[blockIdx.x];
    if (cnt > cap) {
        for (uint32_t b = threadIdx.x; b < G; b += blockDim.x) qseen[b] = 1u;
        return;
    }
    const uint64_t* __restrict__ mine = cand + (int64_t)blockIdx.x * cap;
    for (uint32_t e = threadIdx.x; e < cnt; e += blockDim.x) {
        const uint64_t key = mine[e];
        uint32_t b = bucket_of(key, G);
        for (uint32_t probe = 0; probe < G; ++probe) {
            const uint64_t cur = qkeys[b];
            if (cur == kEmptyKey) break;
            if (cur == key) {
                qseen[b] = 1u;
                break;
            }
            b = (b + 1 == G) ? 0 : b + 1;
        }
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

// One wave per (leader, instance) pair, persistent over the pairs.
__global__ __launch_bounds__(256) void prefix_leaders_kernel(ProbeTables T, int32_t N,
                                                             const int64_t* __restrict__ req_off,
                                                             const uint64_t* __restrict__ req_hashes,
                                                             const int32_t* __restrict__ leaders,
                                                             const uint32_t* __restrict__ n_leaders,
                                                             int32_t* __restrict__ overlap, int closed) {
    const int lane = threadIdx.x & 63;
    const int64_t total = (int64_t)(*n_leaders) * N;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t pair = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); pair < total; pair += waves) {
        const int64_t k = pair / N, i = pair - k * N;
        const int64_t r = leaders[k];
        const int64_t h0 = req_off[r], n = req_off[r + 1] - h0;
        const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
        const bool he = (T.flags[i] & kFlagHasEmptyKey) != 0;
        const int64_t l = closed ? search_run_wave(table, T.nb[i], he, req_hashes + h0, n, lane)
                                 : extend_run_wave(table, T.nb[i], he, req_hashes + h0, n, 0, lane);
        if (lane == 0) overlap[r * N + i] = (int32_t)l;
    }
}

// Leaders, first block: 16 (leader, instance) pairs per wave, four lanes per
// 64-byte bucket.  A pair whose first block is not cached on the instance (most
// pairs) or whose prompt has at most one block is answered here; the others go
// on a list (one atomic per wave) and are extended from block 1 by a wave each.
__global__ __launch_bounds__(256) void leaders_first_kernel(ProbeTables T, int32_t N,
                                                            const int64_t* __restrict__ req_off,
                                                            const uint64_t* __restrict__ req_hashes,
                                                            const int32_t* __restrict__ leaders,
                                                            const uint32_t* __restrict__ n_leaders,
                                                            int32_t* __restrict__ overlap, int64_t* __restrict__ more,
                                                            uint32_t* __restrict__ n_more) {
    const int lane = threadIdx.x & 63, g = lane >> 2, q = lane & 3, shift = 4 * g;
    const int64_t total = (int64_t)(*n_leaders) * N;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t b0 = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 16; b0 < total;
         b0 += waves * 16) {
        const int64_t pair = b0 + g;
        const bool act = pair < total;
        int64_t i = 0, r = 0, h0 = 0, n = 0;
        if (act) {
            const int64_t k = pair / N;
            i = pair - k * N;
            r = leaders[k];
            h0 = req_off[r];
            n = req_off[r + 1] - h0;
        }
        bool hit = false;
        if (act && n > 0) {                              // uniform over the group of four lanes
            const uint64_t key = req_hashes[h0];
            const uint32_t nb = T.nb[i];
            if (key == kEmptyKey) {
                hit = (T.flags[i] & kFlagHasEmptyKey) != 0;
            } else {
                const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
                uint32_t b = bucket_of(key, nb);
                bool gfound = false, gempty = false;
                // a full bucket without the key may have overflowed into the next ones
                for (uint32_t probe = 0; probe < nb && !gfound && !gempty; ++probe) {
                    const ulonglong2 w = *reinterpret_cast<const ulonglong2*>(table + (int64_t)b * kBucketKeys + q * 2);
                    gfound = ((__ballot((w.x == key) | (w.y == key)) >> shift) & 0xFull) != 0;
                    gempty = ((__ballot((w.x == kEmptyKey) | (w.y == kEmptyKey)) >> shift) & 0xFull) != 0;
                    b = (b + 1 == nb) ? 0 : b + 1;
                }
                hit = gfound;
            }
        }
        const bool go_on = act && hit && n > 1;
        if (act && q == 0 && !go_on) overlap[r * N + i] = hit ? 1 : 0;
        const uint64_t m = __ballot(go_on && q == 0);
        if (m) {
            const int first = __ffsll((long long)m) - 1;
            uint32_t base = 0;
            if (lane == first) base = atomicAdd(n_more, (uint32_t)__popcll(m));
            base = (uint32_t)__shfl((int)base, first);
            if (go_on && q == 0) more[base + __popcll(m & ((1ull << lane) - 1))] = pair;
        }
    }
}

// The listed leader pairs, one wave each, from block 1 on.
__global__ __launch_bounds__(256) void leaders_rest_kernel(ProbeTables T, int32_t N,
                                                           const int64_t* __restrict__ req_off,
                                                           const uint64_t* __restrict__ req_hashes,
                                                           const int32_t* __restrict__ leaders,
                                                           const int64_t* __restrict__ more,
                                                           const uint32_t* __restrict__ n_more,
                                                           int32_t* __restrict__ overlap) {
    const int lane = threadIdx.x & 63;
    const int64_t total = *n_more;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t x = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); x < total; x += waves) {
        const int64_t pair = more[x];
        const int64_t k = pair / N, i = pair - k * N;
        const int64_t r = leaders[k];
        const int64_t h0 = req_off[r], n = req_off[r + 1] - h0;
        const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
        const bool he = (T.flags[i] & kFlagHasEmptyKey) != 0;
        const int64_t l = extend_run_wave(table, T.nb[i], he, req_hashes + h0, n, 1, lane, 16);
        if (lane == 0) overlap[r * N + i] = (int32_t)l;
    }
}

// Lane per pair: followers whose answer follows from the leader's (or from a
// continuation cached nowhere) are written here; workgroup b covers pairs
// [b chunk, (b + 1) chunk) and lists the rest in its own slice of the probe
// list (counted in LDS, so no global counter is shared).
constexpr int kResolveThreads = 1024;

// VEC (N a multiple of 4, the overlap matrix 16-byte aligned): a thread takes
// four consecutive instances of one request, reads the leader's four overlaps
// as one 16-byte word and writes its four back as one when all are resolved;
// the chunk is then a multiple of 4.
template <bool VEC>
__global__ __launch_bounds__(kResolveThreads) void followers_resolve_kernel(
    int32_t R, int32_t N, int64_t chunk, const int32_t* __restrict__ lead_of, const int32_t* __restrict__ lcp_of,
    const int32_t* __restrict__ cont_of, const uint32_t* __restrict__ qseen, int32_t* __restrict__ overlap,
    int64_t* __restrict__ list, uint32_t* __restrict__ n_list) {
    constexpr int V = VEC ? 4 : 1;
    __shared__ uint32_t lcount;
    if (threadIdx.x == 0) lcount = 0u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t pairs = (int64_t)R * N;
    const int64_t p_begin = (int64_t)blockIdx.x * chunk;
    const int64_t p_end = p_begin + chunk < pairs ? p_begin + chunk : pairs;
    int64_t* __restrict__ mine = list + p_begin;
    for (int64_t p0 = p_begin; p0 < p_end; p0 += V * kResolveThreads) {
        const int64_t pair = p0 + V * (int64_t)threadIdx.x;
        uint32_t push = 0;                              // bit j: pair + j goes on the probe list
        if (pair < p_end) {
            const int64_t r = pair / N, i = pair - r * N;
            const int64_t lead = lead_of[r];
            if (lead != r) {
                const int32_t c = lcp_of[r];
                const int32_t cont = cont_of[r];
                // the prompt ends in the shared prefix, or block c is cached nowhere
                const bool at_c = cont == kContNone || (cont >= 0 && qseen[cont] == 0u);
                int32_t ll[V], out[V];
                if constexpr (VEC) {
                    const int4 q = *reinterpret_cast<const int4*>(overlap + lead * N + i);
                    ll[0] = q.x; ll[1] = q.y; ll[2] = q.z; ll[3] = q.w;
                } else {
                    ll[0] = overlap[lead * N + i];
                }
#pragma unroll
                for (int j = 0; j < V; ++j) {
                    out[j] = ll[j] < c ? ll[j] : c;
                    if (ll[j] >= c && !at_c) push |= 1u << j;
                }
                if (VEC && push == 0) {
                    *reinterpret_cast<int4*>(overlap + pair) = int4{out[0], out[V > 1 ? 1 : 0], out[V > 2 ? 2 : 0],
                                                                    out[V > 3 ? 3 : 0]};
                } else {
#pragma unroll
                    for (int j = 0; j < V; ++j)
                        if (!((push >> j) & 1u)) overlap[pair + j] = out[j];
                }
            }
        }
        const uint32_t cnt = (uint32_t)__popc(push);
        uint32_t incl = cnt;                            // inclusive scan over the wave
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t up = __shfl_up(incl, d);
            if (lane >= d) incl += up;
        }
        const uint32_t total = __shfl(incl, 63);
        if (total) {
            uint32_t base = 0;
            if (lane == 63) base = atomicAdd(&lcount, total);
            base = (uint32_t)__shfl((int)base, 63) + incl - cnt;
#pragma unroll
            for (int j = 0; j < V; ++j)
                if ((push >> j) & 1u) mine[base++] = pair + j;
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) n_list[blockIdx.x] = lcount;
}

// Block b probes the pairs of slice b, 16 per wave (four lanes per bucket).
__global__ __launch_bounds__(256) void followers_probe_kernel(ProbeTables T, int32_t N, int64_t chunk,
                                                              const int64_t* __restrict__ req_off,
                                                              const uint64_t* __restrict__ req_hashes,
                                                              const int32_t* __restrict__ lcp_of,
                                                              const int64_t* __restrict__ list,
                                                              const uint32_t* __restrict__ n_list,
                                                              int32_t* __restrict__ overlap) {
    const int lane = threadIdx.x & 63;
    const int group = lane >> 2, q = lane & 3, shift = group * 4;
    const int64_t total = n_list[blockIdx.x];
    const int64_t* __restrict__ mine = list + (int64_t)blockIdx.x * chunk;
    for (int64_t w = threadIdx.x >> 6; w * 16 < total; w += blockDim.x >> 6) {
        const int64_t idx = w * 16 + group;
        if (idx >= total) continue;                      // whole group of 4 lanes skips together
        const int64_t pair = mine[idx];
        const int64_t r = pair / N, i = pair - r * N;
        const int64_t h0 = req_off[r], n = req_off[r + 1] - h0;
        const uint64_t* table = T.keys + T.base[i] * kBucketKeys;
        const int64_t l = extend_run(table, T.nb[i], (T.flags[i] & kFlagHasEmptyKey) != 0, req_hashes + h0, n,
                                     lcp_of[r], q, shift);
        if (q == 0) overlap[pair] = (int32_t)l;
    }
}

// Workspace pieces, each starting on a 256-byte boundary.
static inline int64_t ws_round(int64_t b) { return (b + 255) & ~int64_t(255); }
constexpr int64_t kMaxSlices = 8192;     // workgroups of the sliced passes

int64_t prefix_workspace_bytes(int32_t R, int32_t N) {
    const int64_t G = group_table_size(R);
    return 2 * ws_round(G * 8)                  // group table, leader words
           + 5 * ws_round((int64_t)R * 4)       // slot_of, lead_of, lcp_of, leaders, cont_of
           + 256                                // leader counter
           + ws_round(G * 8) + ws_round(G * 4)  // continuation keys, seen flags
           + ws_round((int64_t)kContFilterWords * 4)
           + ws_round(kMaxSlices * 4) + ws_round(kContListCap * 8)   // semi-join candidates
           + ws_round(kMaxSlices * 4) + ws_round((int64_t)R * N * 8);  // probe list
}

bool prefix_use_join(int32_t R, int32_t N, int64_t table_slots, int mode) {
    if (mode == 1) return true;
    if (mode == 2) return false;
    // a random 64-byte probe per follower pair against one sequential pass over every cached key
    return (int64_t)R * N * 4 >= table_slots;
}

hipError_t launch_prefix_match(const CacheTables& t, int32_t R, int32_t N, const int64_t* req_off,
                               const uint64_t* req_hashes, int32_t* overlap, void* workspace, int n_cu,
                               bool join, bool closed, hipStream_t s) {
    const int64_t pairs = (int64_t)R * N;
    if (pairs <= 0) return hipSuccess;
    const int64_t G = group_table_size(R);
    char* p = reinterpret_cast<char*>(workspace);
    auto take = [&](int64_t bytes) {
        char* q = p;
        p += ws_round(bytes);
        return q;
    };
    uint64_t* gkeys = reinterpret_cast<uint64_t*>(take(G * 8));
    unsigned long long* glead = reinterpret_cast<unsigned long long*>(take(G * 8));
    int32_t* slot_of = reinterpret_cast<int32_t*>(take((int64_t)R * 4));
    int32_t* lead_of = reinterpret_cast<int32_t*>(take((int64_t)R * 4));
    int32_t* lcp_of = reinterpret_cast<int32_t*>(take((int64_t)R * 4));
    int32_t* leaders = reinterpret_cast<int32_t*>(take((int64_t)R * 4));
    int32_t* cont_of = reinterpret_cast<int32_t*>(take((int64_t)R * 4));
    uint32_t* n_leaders = reinterpret_cast<uint32_t*>(take(256));
    uint64_t* qkeys = reinterpret_cast<uint64_t*>(take(G * 8));
    uint32_t* qseen = reinterpret_cast<uint32_t*>(take(G * 4));
    uint32_t* n_list = reinterpret_cast<uint32_t*>(take(kMaxSlices * 4));
    uint32_t* qfilter = reinterpret_cast<uint32_t*>(take((int64_t)kContFilterWords * 4));
    uint32_t* n_cand = reinterpret_cast<uint32_t*>(take(kMaxSlices * 4));
    uint64_t* cand = join ? reinterpret_cast<uint64_t*>(take(kContListCap * 8)) : nullptr;
    int64_t* list = reinterpret_cast<int64_t*>(take((int64_t)R * N * 8));

    const int64_t jn = join ? 1 : 0;
    const FillOp fills[6] = {{gkeys, kEmptyKey, G, 8},          {glead, 0u, G, 8},
                             {n_leaders, 0u, 2, 4},              {qkeys, kEmptyKey, jn * G, 8},
                             {qseen, 0u, jn * G, 4},             {qfilter, 0u, jn * kContFilterWords, 4}};
    hipError_t e = launch_fill_multi(fills, 6, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(group_insert_kernel, dim3((uint32_t)(((int64_t)R + kGroupThreads - 1) / kGroupThreads)),
                       dim3(kGroupThreads), 0, s, R, req_off, req_hashes, gkeys, glead, (uint32_t)G, slot_of);
    hipLaunchKernelGGL(group_lcp_kernel, dim3((uint32_t)(((int64_t)R + 15) / 16)), dim3(256), 0, s, R, req_off,
                       req_hashes, glead, slot_of, lead_of, lcp_of, leaders, n_leaders, qkeys, (uint32_t)G, cont_of,
                       join ? 1 : 0);
    if (join) {
        const int64_t n_slots = t.total_buckets * kBucketKeys;
        int64_t grid = (n_slots / 2 + kContThreads - 1) / kContThreads;
        if (grid > n_cu) grid = n_cu;
        if (grid > kMaxSlices) grid = kMaxSlices;
        if (grid < 1) grid = 1;
        hipLaunchKernelGGL(cont_filter_kernel, dim3((uint32_t)((G + 255) / 256)), dim3(256), 0, s, qkeys, (uint32_t)G,
                           qfilter);
        const uint32_t cap = (uint32_t)(kContListCap / grid);
        hipLaunchKernelGGL(cont_scan_kernel, dim3((uint32_t)grid), dim3(kContThreads), 0, s, t.keys, n_slots, qfilter,
                           cand, cap, n_cand);
        hipLaunchKernelGGL(cont_probe_kernel, dim3((uint32_t)grid), dim3(256), 0, s, cand, cap, n_cand, qkeys,
                           (uint32_t)G, qseen);
    }
    ProbeTables T{t.keys, t.base, t.nbuckets, t.flags};
    // leaders: persistent grids of waves over (leader, instance) pairs.  The
    // probe list of the followers is free until they run and holds the leader
    // pairs that go past block 0; n_leaders[1] counts them.
    int64_t wgrid = (pairs + 3) / 4;
    if (wgrid > (int64_t)n_cu * 16) wgrid = (int64_t)n_cu * 16;
    if (closed) {
        hipLaunchKernelGGL(prefix_leaders_kernel, dim3((uint32_t)wgrid), dim3(256), 0, s, T, N, req_off, req_hashes,
                           leaders, n_leaders, overlap, 1);
    } else {
        int64_t fgrid = (pairs + 63) / 64;
        if (fgrid > (int64_t)n_cu * 16) fgrid = (int64_t)n_cu * 16;
        hipLaunchKernelGGL(leaders_first_kernel, dim3((uint32_t)fgrid), dim3(256), 0, s, T, N, req_off, req_hashes,
                           leaders, n_leaders, overlap, list, n_leaders + 1);
        hipLaunchKernelGGL(leaders_rest_kernel, dim3((uint32_t)wgrid), dim3(256), 0, s, T, N, req_off, req_hashes,
                           leaders, list, n_leaders + 1, overlap);
    }
    // followers: slices of pairs, one workgroup each
    const bool vec = N % 4 == 0 && (uintptr_t)overlap % 16 == 0;
    int64_t slices = (pairs + kResolveThreads - 1) / kResolveThreads;
    if (slices > (int64_t)n_cu * 8) slices = (int64_t)n_cu * 8;
    if (slices > kMaxSlices) slices = kMaxSlices;
    int64_t chunk = (pairs + slices - 1) / slices;
    if (vec) chunk = (chunk + 3) & ~int64_t(3);
    slices = (pairs + chunk - 1) / chunk;
    if (vec)
        hipLaunchKernelGGL(followers_resolve_kernel<true>, dim3((uint32_t)slices), dim3(kResolveThreads), 0, s, R, N,
                           chunk, lead_of, lcp_of, cont_of, qseen, overlap, list, n_list);
    else
        hipLaunchKernelGGL(followers_resolve_kernel<false>, dim3((uint32_t)slices), dim3(kResolveThreads), 0, s, R, N,
                           chunk, lead_of, lcp_of, cont_of, qseen, overlap, list, n_list);
    hipLaunchKernelGGL(followers_probe_kernel, dim3((uint32_t)slices), dim3(256), 0, s, T, N, chunk, req_off,
                       req_hashes, lcp_of, list, n_list, overlap);
    return hipGetLastError();
}

}  // namespace ls
