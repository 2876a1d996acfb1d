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
// the 32-bit fingerprints of those continuation hashes in a small table and
// marks, in one sequential pass over the fingerprints of every cached key
// (which each table build leaves behind, 4 bytes per key), the ones some
// instance's key shares (a semi-join).  A follower whose continuation's
// fingerprint is unmarked has its block c cached nowhere, so l[r,i] = c
// wherever l[lead,i] >= c, with no probe; the others are probed.  Two keys that
// share a fingerprint only cost probes, never a wrong overlap.
//
// Probing.  Four lanes share one 64-byte bucket (16 bytes each), so a wave
// probes 16 pairs at once and every probe is one coalesced 64-byte read.  A
// group walks its request's blocks in order and speculatively probes a window
// of consecutive positions that doubles after every all-hit window (1, 2, 4,
// ... kMaxWindow): short runs waste few probes, long runs keep kMaxWindow reads
// in flight.  The first miss ends the pair.
#include <type_traits>

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
// rounds settle an 8k-block prompt.  Exact only under that invariant.  It runs
// on the leader pairs whose first block the first-block pass found cached, from
// block 1 on.
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

// Prefix-closed caches only: the first miss at or after l, given blocks
// [0, l) cached, by galloping (probing l, l + 2, l + 6, l + 14, ... while they
// hit, each hit proving every block before it) and then bisecting between the
// last hit and the miss.  A run of L blocks takes about 2 log2(L) probes
// instead of about L / 8 rounds of the walk.  All four lanes of a group call it
// together (group-wide ballots).
__device__ __forceinline__ int64_t gallop_run(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                              const uint64_t* __restrict__ h, int64_t n, int64_t l, int q,
                                              int shift) {
    int64_t lo = l, hi = n;                      // blocks [0, lo) cached; block hi missing (or hi = n)
    for (int64_t step = 1; lo < hi; step *= 2) {
        const int64_t j = lo + step - 1 < hi ? lo + step - 1 : hi - 1;
        if (!probe_block(table, nb, has_empty, h[j], q, shift)) {
            hi = j;
            break;
        }
        lo = j + 1;
    }
    while (lo < hi) {
        const int64_t j = lo + (hi - lo) / 2;
        if (probe_block(table, nb, has_empty, h[j], q, shift)) lo = j + 1;
        else hi = j;
    }
    return lo;
}

// `start`: blocks [0, start) are known to be cached.
__device__ __forceinline__ int64_t search_run_wave(const uint64_t* __restrict__ table, uint32_t nb, bool has_empty,
                                                   const uint64_t* __restrict__ h, int64_t n, int64_t start,
                                                   int lane) {
    const int g = lane >> 2, q = lane & 3, shift = g * 4;
    int64_t lo = start, hi = n;                  // blocks [0, lo) cached; block hi is the first miss (or n)
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

// Continuation table: open addressing over G slots (a power of two, at most
// half full) of fingerprints, kFpEmpty marking an empty slot.  The thread that
// claims a slot also sets the fingerprint's three bits in the scan's filter, a
// Bloom filter blocked by 32-bit word: word f >> 17, bits f & 31, (f >> 5) & 31
// and (f >> 10) & 31, so a test is one word read and a few bit operations
// (about 0.6 % of other fingerprints pass at 65,536 continuations).
constexpr int kContFilterLog = 20;
constexpr int kContFilterWords = (1 << kContFilterLog) / 32;     // 128 KiB
static_assert(kContFilterWords == 1 << 15, "the filter word is the fingerprint's top 15 bits");

__device__ __forceinline__ uint32_t fp_slot(uint32_t f, uint32_t G) {
    return (uint32_t)(((uint64_t)(f * 0x85EBCA77u) * G) >> 32);
}

__device__ __forceinline__ uint32_t fp_word_bits(uint32_t f) {
    return (1u << (f & 31)) | (1u << ((f >> 5) & 31)) | (1u << ((f >> 10) & 31));
}

__device__ __forceinline__ int32_t cont_insert(uint32_t* __restrict__ qfp, uint32_t G, uint32_t f,
                                               uint32_t* __restrict__ filter) {
    uint32_t b = fp_slot(f, G);
    for (uint32_t probe = 0; probe < G; ++probe) {
        const uint32_t cur = qfp[b];
        if (cur == f) return (int32_t)b;
        if (cur == kFpEmpty) {
            const uint32_t old = atomicCAS(qfp + b, kFpEmpty, f);
            if (old == kFpEmpty) {
                atomicOr(&filter[f >> 17], fp_word_bits(f));
                return (int32_t)b;
            }
            if (old == f) return (int32_t)b;
        }
        b = (b + 1 == G) ? 0 : b + 1;
    }
    return kContProbe;
}

// What the semi-join found for a continuation slot: qseen counts the matches,
// and the first kSeenInst of them record their instance in qinst (a 16-byte
// word per slot).  0: the continuation's block is cached nowhere; 1 ..
// kSeenInst: at most on the recorded instances; more: on any instance.  A
// nonzero qall (the build's key listing incomplete, or a candidate list
// overflowed) makes every continuation count as cached on any instance.
constexpr uint32_t kSeenInst = 4;
constexpr uint32_t kSeenAny = kSeenInst + 1;

// One wave per request: leader id and common-prefix length with the leader;
// leaders append themselves to the leader list.  With the semi-join on, a
// follower registers the fingerprint of its block c (cont_of: slot, kContNone
// when c reaches its end, kContProbe when it must be probed).
template <int LPR>
__global__ __launch_bounds__(256) void group_lcp_kernel(int32_t R, const int64_t* __restrict__ req_off,
                                                        const uint64_t* __restrict__ req_hashes,
                                                        const unsigned long long* __restrict__ glead,
                                                        const int32_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ lead_of, int32_t* __restrict__ lcp_of,
                                                        int32_t* __restrict__ leaders, uint32_t* __restrict__ n_leaders,
                                                        uint32_t* __restrict__ qfp, uint32_t G,
                                                        uint32_t* __restrict__ qfilter, int32_t* __restrict__ cont_of,
                                                        int join) {
    // LPR lanes per request (16: four requests per wave, for large batches,
    // where more requests in flight pay; 64: a wave per request, for small
    // batches of long prompts, where the rounds of one request are the cost).
    // A round compares LPR w positions, lane sl taking j0 + sl + LPR u (u < w),
    // all loads issued before any compare; w doubles after every all-equal
    // round (1, 2, 4, 8), so long common prefixes take few dependent rounds.
    static_assert(LPR == 16 || LPR == 64, "a request's lanes share one wave");
    constexpr int kLcpMaxLoads = 8;
    const int lane = threadIdx.x & 63, sg = lane / LPR, sl = lane % LPR;
    const int64_t r = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * (64 / LPR) + sg;
    if (r >= R) return;                               // uniform over the request's lanes
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
        for (int64_t j0 = 0; j0 < m; j0 += LPR * w, w = w * 2 > kLcpMaxLoads ? kLcpMaxLoads : w * 2) {
            uint64_t av[kLcpMaxLoads], bv[kLcpMaxLoads];
#pragma unroll
            for (int u = 0; u < kLcpMaxLoads; ++u) {
                const int64_t j = j0 + sl + LPR * u;
                if (u < w && j < m) {
                    av[u] = a[j];
                    bv[u] = b[j];
                }
            }
            int64_t first = m;                       // this lane's first differing position
#pragma unroll
            for (int u = kLcpMaxLoads - 1; u >= 0; --u) {
                const int64_t j = j0 + sl + LPR * u;
                if (u < w && j < m && av[u] != bv[u]) first = j;
            }
#pragma unroll
            for (int off = LPR / 2; off >= 1; off >>= 1) {
                const int64_t o = __shfl_xor(first, off, LPR);
                first = o < first ? o : first;
            }
            if (first < m) {                          // uniform over the request's lanes
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
            cont = (join && key != kEmptyKey) ? cont_insert(qfp, G, key_fp(key), qfilter) : kContProbe;
        }
        cont_of[r] = cont;
    }
}

// The semi-join pass: every cached key's fingerprint looks itself up among the
// continuations'.  The continuations' Bloom filter sits in LDS, so the pass
// streams the fingerprint runs of the table build and tests one LDS word per
// key.  The positions of the fingerprints that pass go on a list of the wave's
// own in LDS, which the wave looks up in the continuation table whenever it
// holds kWaveFlush or more and at the end (a wave whose list overflows makes
// every continuation count as cached everywhere).  A match records its instance with the
// continuation: the follower is then probed on the recorded instances only.
// Waves take whole segments and run unsynchronised after the filter copy, so
// the tests and lookups of some overlap the loads of others.  If the build
// could not list every key that went through its overflow pass, every
// continuation counts as cached everywhere (its followers are probed, so the
// overlaps stay exact).
constexpr int kContThreads = 1024;
constexpr int kContWaves = kContThreads / 64;
constexpr int kContLoads = 8;                      // 16-byte loads per lane per chunk
constexpr uint32_t kContChunk = 64 * 4 * kContLoads;   // fingerprints per chunk of a wave (2048)
constexpr uint32_t kWaveCand = 512;                // LDS candidate list of each wave: positions (2 KiB)
constexpr uint32_t kWaveFlush = 256;               // a wave looks its list up once it holds this many
constexpr uint32_t kExtraTag = 0x80000000u;        // list entry of the overflow pass's list

__device__ __forceinline__ void cont_mark(const uint32_t* __restrict__ qfp, uint32_t G, uint32_t f, uint32_t inst,
                                          uint32_t* __restrict__ qseen, uint32_t* __restrict__ qinst) {
    uint32_t b = fp_slot(f, G);
    for (uint32_t probe = 0; probe < G; ++probe) {
        const uint32_t cur = qfp[b];
        if (cur == kFpEmpty) return;
        if (cur == f) {
            if (qseen[b] > kSeenInst) return;             // already unlimited
            const uint32_t k = atomicAdd(qseen + b, 1u);
            if (k < kSeenInst) qinst[(int64_t)b * kSeenInst + k] = inst;
            return;
        }
        b = (b + 1 == G) ? 0 : b + 1;
    }
}

__global__ __launch_bounds__(kContThreads) void cont_scan_kernel(
    const uint32_t* __restrict__ fp, const uint32_t* __restrict__ fp_len, const uint32_t* __restrict__ fp_inst,
    int32_t n_seg, const uint32_t* __restrict__ fp_extra, const uint32_t* __restrict__ fp_extra_inst,
    const uint32_t* __restrict__ fp_meta, uint32_t fp_extra_cap, const uint32_t* __restrict__ filter,
    const uint32_t* __restrict__ qfp, uint32_t G, uint32_t* __restrict__ qseen, uint32_t* __restrict__ qinst,
    uint32_t* __restrict__ qall) {
    __shared__ uint32_t lf[kContFilterWords];
    __shared__ uint32_t cand[kContWaves][kWaveCand];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const uint32_t n_extra = fp_meta[0];
    if (n_extra > fp_extra_cap) {                         // uniform: some cached keys are listed nowhere
        if (blockIdx.x == 0 && tid == 0) qall[0] = 1u;
        return;
    }
    uint32_t* __restrict__ mine = cand[wv];
    uint32_t wcount = 0;                                  // entries of this wave's list (uniform)
    // looks the wave's listed candidates up in the continuation table; an
    // entry is the fingerprint's position in the runs, or kExtraTag | j for
    // entry j of the overflow pass's list
    auto flush = [&]() {
        for (uint32_t e = (uint32_t)lane; e < wcount; e += 64) {
            const uint32_t p = mine[e];
            uint32_t f, inst;
            if (p & kExtraTag) {
                f = fp_extra[p & ~kExtraTag];
                inst = fp_extra_inst[p & ~kExtraTag];
            } else {
                f = fp[p];
                inst = fp_inst[p / (uint32_t)kSegSlots];
            }
            cont_mark(qfp, G, f, inst, qseen, qinst);
        }
        wcount = 0;
    };
    // appends the entries pos + k of the lanes whose bit is set in the ballot
    // m[k] (K of them) to the wave's list: entry k of a lane goes after the
    // wave's entries of slots below k and the lanes below it (lane-mask
    // counts).  A list that overflows drops the rest and sets qall, which
    // makes every continuation count as cached on every instance.  Every lane
    // of the wave calls it, and only when some lane hit.
    auto append = [&](const uint64_t* m, uint32_t pos, int K) {
        uint32_t at0 = wcount;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if ((m[k] >> lane) & 1ull) {
                const uint32_t at = at0 + __builtin_amdgcn_mbcnt_hi((uint32_t)(m[k] >> 32),
                                                                    __builtin_amdgcn_mbcnt_lo((uint32_t)m[k], 0u));
                if (at < kWaveCand) mine[at] = pos + (uint32_t)k;
            }
            at0 += (uint32_t)__popcll(m[k]);
        }
        if (at0 > kWaveCand) {                            // uniform
            if (lane == 0) qall[0] = 1u;
            at0 = kWaveCand;
        }
        wcount = at0;
    };
    // tests four fingerprints of a lane, at positions e0 .. e0 + 3 of segment
    // L's run of len (FULL: the wave's whole group lies inside the run); the
    // LDS reads go out together and each test is a ballot
    auto test4 = [&](auto full_tag, const uint4& x, uint32_t e0, uint32_t len, uint32_t run0) {
        constexpr bool FULL = decltype(full_tag)::value;
        const uint32_t f[4] = {x.x, x.y, x.z, x.w};
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = lf[f[k] >> 17];
        uint64_t m[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t bits = fp_word_bits(f[k]);
            if constexpr (FULL) m[k] = __ballot((w[k] & bits) == bits);
            else m[k] = __ballot(((w[k] & bits) == bits) & (e0 + (uint32_t)k < len));
        }
        if ((m[0] | m[1] | m[2] | m[3]) != 0) append(m, run0 + e0, 4);   // uniform over the wave
    };
    // The wave's chunks: segments w, w + W, ... of the grid's W waves, each in
    // chunks of kContChunk fingerprints.  Two chunk buffers (A, B) alternate:
    // a chunk's loads go out before the chunk ahead of it is tested, and the
    // first two go out before the filter copy.  The cursor is uniform over the
    // wave, and no barrier ties the waves together after the copy.
    struct Chunk {
        uint32_t c0, len;
        int64_t L;
        bool on;
    };
    const int64_t W = (int64_t)gridDim.x * kContWaves;
    int64_t cur_L = (int64_t)blockIdx.x * kContWaves + wv;
    uint32_t cur_c0 = 0, cur_len = cur_L < n_seg ? fp_len[cur_L] : 0u;
    auto take = [&](Chunk& d) {
        d.on = cur_L < n_seg;
        if (!d.on) {
            d.L = 0;
            d.c0 = 0;
            d.len = 0;
            return;
        }
        d.L = cur_L;
        d.c0 = cur_c0;
        d.len = cur_len;
        cur_c0 += kContChunk;
        if (cur_c0 >= cur_len) {
            cur_L += W;
            cur_c0 = 0;
            cur_len = cur_L < n_seg ? fp_len[cur_L] : 0u;
        }
    };
    // Every lane issues all kContLoads loads of a chunk, so that each refill is
    // the same straight run of loads and a test waits only for its own buffer.
    // They stay inside the segment's slots: c0 is a multiple of kContChunk
    // below len <= kSegSlots, so e < kSegSlots; past len (or, with no chunk,
    // in segment 0) they read data the test ignores.
    static_assert(kSegSlots % kContChunk == 0, "chunks tile a segment's slots");
    auto load = [&](const Chunk& d, uint4 (&x)[kContLoads]) {
        const uint4* __restrict__ run = reinterpret_cast<const uint4*>(fp + d.L * kSegSlots);
#pragma unroll
        for (int u = 0; u < kContLoads; ++u) x[u] = run[d.c0 / 4 + (uint32_t)(lane + 64 * u)];
    };
    // a group of four past the run's end for the whole wave is skipped, one
    // inside it for the whole wave is tested without the bound; the wave looks
    // its list up when it holds kWaveFlush entries or more
    auto test_chunk = [&](const Chunk& d, const uint4 (&x)[kContLoads]) {
        const uint32_t run0 = (uint32_t)(d.L * kSegSlots);
        if (d.c0 + kContChunk <= d.len) {                // uniform: the whole chunk lies inside the run
#pragma unroll
            for (int u = 0; u < kContLoads; ++u)
                test4(std::true_type{}, x[u], d.c0 + 4u * (uint32_t)(lane + 64 * u), d.len, run0);
        } else {
#pragma unroll
            for (int u = 0; u < kContLoads; ++u) {
                const uint32_t first = d.c0 + 256u * (uint32_t)u;
                if (first < d.len) test4(std::false_type{}, x[u], d.c0 + 4u * (uint32_t)(lane + 64 * u), d.len, run0);
            }
        }
        if (wcount >= kWaveFlush) flush();
    };
    Chunk da, db;
    uint4 xa[kContLoads], xb[kContLoads];
    take(da);
    load(da, xa);
    take(db);
    load(db, xb);
    {
        const uint4* __restrict__ f4 = reinterpret_cast<const uint4*>(filter);
        uint4* l4 = reinterpret_cast<uint4*>(lf);
        for (int e = tid; e < kContFilterWords / 4; e += kContThreads) l4[e] = f4[e];
    }
    __syncthreads();
    while (da.on || db.on) {                              // uniform over the wave
        test_chunk(da, xa);                               // nothing to test without a chunk (len 0)
        take(da);
        load(da, xa);
        test_chunk(db, xb);
        take(db);
        load(db, xb);
    }
    // the keys of the overflow pass, 64 per wave of the grid
    for (int64_t j0 = ((int64_t)blockIdx.x * kContWaves + wv) * 64; j0 < n_extra; j0 += W * 64) {
        const int64_t j = j0 + lane;
        bool hit = false;
        if (j < n_extra) {
            const uint32_t f = fp_extra[j];
            const uint32_t bits = fp_word_bits(f);
            hit = f != kFpEmpty && (lf[f >> 17] & bits) == bits;
        }
        const uint64_t m[1] = {__ballot(hit)};
        if (m[0] != 0) append(m, kExtraTag | (uint32_t)j, 1);
        if (wcount >= kWaveFlush) flush();
    }
    flush();
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

// Leaders, first block: 16 (leader, instance) pairs per wave, four lanes per
// 64-byte bucket.  A pair whose first block is not cached on the instance (most
// pairs) or whose prompt has at most one block is answered here; the others go
// on a list and are extended from block 1 by a wave each.  The workgroup's
// waves step through the pairs together, kLeadThreads / 4 per round, and a
// round's list entries are counted in LDS and claimed with one global add:
// adds to one global counter from every wave serialise.
constexpr int kLeadThreads = 1024;
constexpr int64_t kLeadPairs = kLeadThreads / 4;

__global__ __launch_bounds__(kLeadThreads) void leaders_first_kernel(ProbeTables T, int32_t N,
                                                                     const int64_t* __restrict__ req_off,
                                                                     const uint64_t* __restrict__ req_hashes,
                                                                     const int32_t* __restrict__ leaders,
                                                                     const uint32_t* __restrict__ n_leaders,
                                                                     int32_t* __restrict__ overlap,
                                                                     int64_t* __restrict__ more,
                                                                     uint32_t* __restrict__ n_more) {
    __shared__ uint32_t lcount, lbase;
    const int lane = threadIdx.x & 63, g = lane >> 2, q = lane & 3, shift = 4 * g;
    const int64_t total = (int64_t)(*n_leaders) * N;
    for (int64_t r0 = (int64_t)blockIdx.x * kLeadPairs; r0 < total; r0 += (int64_t)gridDim.x * kLeadPairs) {
        if (threadIdx.x == 0) lcount = 0u;
        __syncthreads();
        const int64_t pair = r0 + (threadIdx.x >> 2);
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
        uint32_t wbase = 0;
        if (m != 0 && lane == __ffsll((long long)m) - 1) wbase = atomicAdd(&lcount, (uint32_t)__popcll(m));
        __syncthreads();
        if (threadIdx.x == 0) lbase = lcount ? atomicAdd(n_more, lcount) : 0u;
        __syncthreads();
        if (m != 0) {
            wbase = lbase + (uint32_t)__shfl((int)wbase, __ffsll((long long)m) - 1);
            if (go_on && q == 0) more[wbase + __popcll(m & ((1ull << lane) - 1))] = pair;
        }
        __syncthreads();                                  // lcount and lbase are reused next round
    }
}

// The listed leader pairs, one wave each, from block 1 on: walked, or with
// prefix-closed caches (`closed`) searched for the run's end.
__global__ __launch_bounds__(256) void leaders_rest_kernel(ProbeTables T, int32_t N,
                                                           const int64_t* __restrict__ req_off,
                                                           const uint64_t* __restrict__ req_hashes,
                                                           const int32_t* __restrict__ leaders,
                                                           const int64_t* __restrict__ more,
                                                           const uint32_t* __restrict__ n_more,
                                                           int32_t* __restrict__ overlap, int closed) {
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
        const int64_t l = closed ? search_run_wave(table, T.nb[i], he, req_hashes + h0, n, 1, lane)
                                 : extend_run_wave(table, T.nb[i], he, req_hashes + h0, n, 1, lane, 16);
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
    const int32_t* __restrict__ cont_of, const uint32_t* __restrict__ qseen, const uint4* __restrict__ qinst,
    const uint32_t* __restrict__ qall, int32_t* __restrict__ overlap, int64_t* __restrict__ list,
    uint32_t* __restrict__ n_list) {
    constexpr int V = VEC ? 4 : 1;
    __shared__ uint32_t lcount;
    if (threadIdx.x == 0) lcount = 0u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const bool any_inst = qall[0] != 0u;                 // every continuation may be cached anywhere
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
                const uint32_t seen = cont < 0 || any_inst ? kSeenAny : qseen[cont];
                // the prompt ends in the shared prefix, or block c is cached nowhere
                const bool at_c = cont == kContNone || seen == 0u;
                // the instances that may hold block c, when the semi-join recorded them all
                uint4 holders = {~0u, ~0u, ~0u, ~0u};
                if (!at_c && seen <= kSeenInst) holders = qinst[cont];
                auto may_hold = [&](uint32_t inst) -> bool {
                    if (seen > kSeenInst) return true;
                    return (holders.x == inst) | (seen > 1u && holders.y == inst) | (seen > 2u && holders.z == inst) |
                           (seen > 3u && holders.w == inst);
                };
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
                    // block c may be cached on this instance: probe it
                    if (ll[j] >= c && !at_c && may_hold((uint32_t)(i + j))) push |= 1u << j;
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

// Block b probes the pairs of slice b, 16 per wave (four lanes per bucket),
// walking from the common prefix, or with prefix-closed caches (`closed`)
// galloping from it.
__global__ __launch_bounds__(256) void followers_probe_kernel(ProbeTables T, int32_t N, int64_t chunk,
                                                              const int64_t* __restrict__ req_off,
                                                              const uint64_t* __restrict__ req_hashes,
                                                              const int32_t* __restrict__ lcp_of,
                                                              const int64_t* __restrict__ list,
                                                              const uint32_t* __restrict__ n_list,
                                                              int32_t* __restrict__ overlap, int closed) {
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
        const bool he = (T.flags[i] & kFlagHasEmptyKey) != 0;
        const int64_t l = closed ? gallop_run(table, T.nb[i], he, req_hashes + h0, n, lcp_of[r], q, shift)
                                 : extend_run(table, T.nb[i], he, req_hashes + h0, n, lcp_of[r], q, shift);
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
           + 2 * ws_round(G * 4)                // continuation fingerprints, seen flags
           + ws_round(G * 16)                   // instances recorded per continuation
           + ws_round((int64_t)kContFilterWords * 4)
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
    uint32_t* qfp = reinterpret_cast<uint32_t*>(take(G * 4));
    uint32_t* qseen = reinterpret_cast<uint32_t*>(take(G * 4));
    uint32_t* qinst = reinterpret_cast<uint32_t*>(take(G * 16));
    uint32_t* n_list = reinterpret_cast<uint32_t*>(take(kMaxSlices * 4));
    uint32_t* qfilter = reinterpret_cast<uint32_t*>(take((int64_t)kContFilterWords * 4));
    int64_t* list = reinterpret_cast<int64_t*>(take((int64_t)R * N * 8));

    if (join && (!t.fp || !t.fp_len || !t.fp_inst || !t.fp_extra || !t.fp_extra_inst || !t.fp_meta))
        return hipErrorInvalidValue;
    // the semi-join's lists hold 31-bit positions: tables of 2^31 slots or more go without it
    if ((int64_t)t.n_seg * kSegSlots > (int64_t)kExtraTag || t.fp_extra_cap >= (int64_t)kExtraTag) join = false;
    const int64_t jn = join ? 1 : 0;
    uint32_t* qall = n_leaders + 2;                // leader counters, then the semi-join's flag
    const FillOp fills[6] = {{gkeys, kEmptyKey, G, 8},          {glead, 0u, G, 8},
                             {n_leaders, 0u, 3, 4},              {qfp, kFpEmpty, jn * G, 4},
                             {qseen, 0u, jn * G, 4},             {qfilter, 0u, jn * kContFilterWords, 4}};
    hipError_t e = launch_fill_multi(fills, 6, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(group_insert_kernel, dim3((uint32_t)(((int64_t)R + kGroupThreads - 1) / kGroupThreads)),
                       dim3(kGroupThreads), 0, s, R, req_off, req_hashes, gkeys, glead, (uint32_t)G, slot_of);
    // a wave per request when the batch leaves most of the device idle at four per wave
    if ((int64_t)R * 16 < (int64_t)n_cu * 256)
        hipLaunchKernelGGL(group_lcp_kernel<64>, dim3((uint32_t)(((int64_t)R + 3) / 4)), dim3(256), 0, s, R, req_off,
                           req_hashes, glead, slot_of, lead_of, lcp_of, leaders, n_leaders, qfp, (uint32_t)G, qfilter,
                           cont_of, join ? 1 : 0);
    else
        hipLaunchKernelGGL(group_lcp_kernel<16>, dim3((uint32_t)(((int64_t)R + 15) / 16)), dim3(256), 0, s, R,
                           req_off, req_hashes, glead, slot_of, lead_of, lcp_of, leaders, n_leaders, qfp, (uint32_t)G,
                           qfilter, cont_of, join ? 1 : 0);
    if (join) {
        // a wave per segment, up to a workgroup per compute unit
        int64_t grid = ((int64_t)t.n_seg + kContWaves - 1) / kContWaves;
        if (grid > n_cu) grid = n_cu;
        if (grid < 1) grid = 1;
        const uint32_t xcap = (uint32_t)(t.fp_extra_cap < 0xFFFFFFFFll ? t.fp_extra_cap : 0xFFFFFFFEll);
        hipLaunchKernelGGL(cont_scan_kernel, dim3((uint32_t)grid), dim3(kContThreads), 0, s, t.fp, t.fp_len,
                           t.fp_inst, t.n_seg, t.fp_extra, t.fp_extra_inst, t.fp_meta, xcap, qfilter, qfp,
                           (uint32_t)G, qseen, qinst, qall);
    }
    ProbeTables T{t.keys, t.base, t.nbuckets, t.flags};
    // leaders: persistent grids of waves over (leader, instance) pairs.  The
    // probe list of the followers is free until they run and holds the leader
    // pairs that go past block 0; n_leaders[1] counts them.
    int64_t wgrid = (pairs + 3) / 4;
    if (wgrid > (int64_t)n_cu * 16) wgrid = (int64_t)n_cu * 16;
    {
        // pairs <= R N bound the leader pairs; every round of a workgroup takes kLeadPairs
        int64_t fgrid = (pairs + kLeadPairs - 1) / kLeadPairs;
        if (fgrid > (int64_t)n_cu * 4) fgrid = (int64_t)n_cu * 4;
        hipLaunchKernelGGL(leaders_first_kernel, dim3((uint32_t)fgrid), dim3(kLeadThreads), 0, s, T, N, req_off,
                           req_hashes, leaders, n_leaders, overlap, list, n_leaders + 1);
        hipLaunchKernelGGL(leaders_rest_kernel, dim3((uint32_t)wgrid), dim3(256), 0, s, T, N, req_off, req_hashes,
                           leaders, list, n_leaders + 1, overlap, closed ? 1 : 0);
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
                           chunk, lead_of, lcp_of, cont_of, qseen, reinterpret_cast<const uint4*>(qinst), qall, overlap, list,
                           n_list);
    else
        hipLaunchKernelGGL(followers_resolve_kernel<false>, dim3((uint32_t)slices), dim3(kResolveThreads), 0, s, R, N,
                           chunk, lead_of, lcp_of, cont_of, qseen, reinterpret_cast<const uint4*>(qinst), qall, overlap, list,
                           n_list);
    hipLaunchKernelGGL(followers_probe_kernel, dim3((uint32_t)slices), dim3(256), 0, s, T, N, chunk, req_off,
                       req_hashes, lcp_of, list, n_list, overlap, closed ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ls
