// Internal declarations shared by the HIP sources of liblodestar.
// Nothing here is part of the C ABI (include/lodestar.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "lodestar.h"

namespace ls {

// ---------------------------------------------------------------------------
// Prefix-cache hash tables.  One open-addressing table per instance; a bucket
// is 8 uint64 keys (64 bytes, one HBM burst).  Empty slots hold kEmptyKey; the
// key kEmptyKey itself is recorded in a per-instance flag instead.
// ---------------------------------------------------------------------------
constexpr int kBucketKeys = 8;
constexpr uint64_t kEmptyKey = ~0ull;
constexpr uint32_t kFlagHasEmptyKey = 1u;

struct CacheTables {
    uint64_t* keys = nullptr;        // [total_buckets * kBucketKeys]
    int64_t* base = nullptr;         // [N] first bucket of instance i
    uint32_t* nbuckets = nullptr;    // [N]
    uint32_t* flags = nullptr;       // [N]
    int32_t n = 0;
    int64_t total_buckets = 0;
    // Fingerprints (key_fp) of every cached key, written by each build for the
    // prefix pass's semi-join: segment L's keys at fp[L * kSegBuckets *
    // kBucketKeys], fp_len[L] of them, all of instance fp_inst[L]; the keys the
    // overflow pass inserted in fp_extra, with their instances in
    // fp_extra_inst, their count in fp_meta[0] (a count above fp_extra_cap
    // means they are not all listed).
    uint32_t* fp = nullptr;
    uint32_t* fp_len = nullptr;      // [n_seg]
    uint32_t* fp_inst = nullptr;     // [n_seg]
    uint32_t* fp_extra = nullptr;    // [fp_extra_cap]
    uint32_t* fp_extra_inst = nullptr;
    uint32_t* fp_meta = nullptr;     // [1]
    int64_t fp_extra_cap = 0;
    int32_t n_seg = 0;
};

// A 32-bit fingerprint of a block hash: the high word of a multiplicative hash
// (independent of bucket_of's), never the all-ones word, which marks an empty
// slot of the tables that hold fingerprints.  Distinct keys may share one.
constexpr uint32_t kFpEmpty = 0xFFFFFFFFu;
__host__ __device__ inline uint32_t key_fp(uint64_t key) {
    const uint32_t f = (uint32_t)((key * 0xD6E8FEB86659FD93ull) >> 32);
    return f == kFpEmpty ? kFpEmpty - 1u : f;
}

// Bucket of `key` in a table of nb buckets: Fibonacci hashing of the whole key,
// high 32 bits mapped onto [0, nb) by a multiply-shift.
__host__ __device__ inline uint32_t bucket_of(uint64_t key, uint32_t nb) {
    uint64_t h = key * 0x9E3779B97F4A7C15ull;
    return (uint32_t)(((h >> 32) * (uint64_t)nb) >> 32);
}

// ---------------------------------------------------------------------------
// Model layout on the device.  Masters are fp32 in the ABI packing.  The
// "compute copy" is what the kernels read: weights rounded to bf16 in LS_BF16
// mode (kept as fp32 values), with layer 2 transposed so that a fixed input k
// addresses consecutive output units.
// ---------------------------------------------------------------------------
struct ModelDims {
    int d = 0, d_inst = 0, h1 = 0, h2 = 0;   // h1, h2: the two hidden widths of a two-layer model
    int L = 2;                                // hidden layers, 1..3
    int h[3] = {0, 0, 0};                     // hidden widths
    int hl = 0;                               // width of the last hidden layer
    bool bf16 = false;
    bool mfma_chains = true;                  // canonical chains on the matrix cores where the batch fills the device
    int block_tokens = 16;
    // master offsets (floats), the ABI packing: per layer W [out x in] then b [out]
    int64_t m_w1 = 0, m_b1 = 0, m_w2 = 0, m_b2 = 0, m_w3 = 0, m_b3 = 0, n_params = 0;   // two-layer names
    int64_t m_w[4] = {0, 0, 0, 0}, m_b[4] = {0, 0, 0, 0};                            // layer l = 0..L (L: head)
    // compute-copy offsets (floats).  Two-layer layout (the fused scorers):
    int64_t c_w1 = 0;   // [h1 x d]  row-major (W1[k][c])
    int64_t c_b1 = 0;   // [h1]
    int64_t c_w2t = 0;  // [h1 x h2] W2T[k][j] = W2[j][k]
    int64_t c_b2 = 0;   // [h2]
    int64_t c_w3 = 0;   // [h2]
    int64_t c_b3 = 0;   // [1]
    int64_t c_w1t = 0;  // [d x h1]  W1T[c][k] = W1[k][c]  (update forward)
    // every depth: layer l's transposed weights W_l^T [in x out] and bias (for
    // two layers these alias the arrays above)
    int64_t c_wt[4] = {0, 0, 0, 0}, c_bl[4] = {0, 0, 0, 0};
    int64_t n_compute = 0;
    int in_of(int l) const { return l == 0 ? d : h[l - 1]; }
    int out_of(int l) const { return l == L ? 1 : h[l]; }
};

// Dropout while training (one update call): inverted dropout on the hidden
// activations, off when thr53 = 0.  Unit j of hidden layer l for row b draws
// splitmix64 output c + 1 for `seed`, c = ((step * 4 + l) * 2^24 + b) * 2^10 + j,
// and is dropped when the draw's top 53 bits are below thr53 = floor(p 2^53);
// a kept unit is multiplied by `scale` = the fp32 value of 1 / (1 - p).
struct DropArgs {
    uint64_t seed = 0, step = 0, thr53 = 0;
    float scale = 1.0f;
};

ModelDims make_dims(const ls_model_config& cfg);

// bf16 matrix-core path: fragment tables derived from the masters.
// frag16 (bf16 bits): W1 [4][h1/32] fragments, W2 [h2/32][h1/16] fragments and
// head fragments [h2/16] (rows w3 and |w3|); a fragment is 64 lanes x 8 bf16.
// frag32: b1 then b2 as [tile][lane half][16].
// Fragment tables of the matrix-core scorer (bf16 part frag16, fp32 part frag32):
//   W1 tail  one A fragment per layer-1 row tile, the 5 derived columns only
//            (the instance columns are resumed from the per-instance partials)
//   W2       A fragments [row tile][k-step]
//   head     per k-step and lane half, the 8 inputs of rows w3 and |w3|
//   b2       the layer-2 biases (fp32)
struct MfmaLayout {
    int d = 0, d_inst = 0, h1 = 0, h2 = 0;
    int64_t m_w1 = 0, m_b1 = 0, m_w2 = 0, m_b2 = 0, m_w3 = 0;
    int64_t w1_frags = 0, w2_frags = 0, n_head = 0, n16 = 0, n32 = 0;
};

inline MfmaLayout make_mfma_layout(const ModelDims& m) {
    MfmaLayout L;
    L.d = m.d; L.d_inst = m.d_inst; L.h1 = m.h1; L.h2 = m.h2;
    L.m_w1 = m.m_w1; L.m_b1 = m.m_b1; L.m_w2 = m.m_w2; L.m_b2 = m.m_b2; L.m_w3 = m.m_w3;
    L.w1_frags = m.h1 / 32;
    L.w2_frags = (int64_t)(m.h2 / 32) * (m.h1 / 16);
    L.n_head = (int64_t)(m.h2 / 16) * 32;
    L.n16 = (L.w1_frags + L.w2_frags) * 512 + L.n_head;
    L.n32 = m.h2;
    return L;
}

// Half-width of the candidate band around each fast bf16 score, relative to
// sum_j |w3_j| h2_j + |b3| (the magnitude the head sums).
constexpr float kBandRel = 0x1p-7f;

bool mfma_supported(const ModelDims& m);

// ---------------------------------------------------------------------------
// Kernel launchers (each returns hipGetLastError() of its launch).
// ---------------------------------------------------------------------------
hipError_t launch_fill_u64(uint64_t* p, uint64_t value, int64_t count, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t count, hipStream_t s);
// Several fills in one launch (4- or 8-byte words; at most kMaxFillOps).
struct FillOp {
    void* p;
    uint64_t value;
    int64_t count;
    int bytes;
};
constexpr int kMaxFillOps = 8;
hipError_t launch_fill_multi(const FillOp* ops, int n, hipStream_t s);
// Table build: the keys partitioned by segment of kSegBuckets buckets (seg_off[i]
// is the first segment of instance i, n_seg the total), one workgroup per
// segment, then a global pass over the keys that overflowed their segment.  The
// workspace (table_build_workspace_bytes) holds the partition and an overflow
// queue of table_overflow_capacity(total) key indices; key indices are 32-bit.
constexpr uint32_t kSegBuckets = 2048;
constexpr int64_t kSegSlots = (int64_t)kSegBuckets * kBucketKeys;
int64_t table_overflow_capacity(int64_t total);
// Bytes of the fingerprint buffer for n_seg segments and an overflow list of
// extra_cap keys, and its carving into t's fp fields.
int64_t table_fp_bytes(int32_t n_seg, int64_t extra_cap);
void carve_table_fp(CacheTables& t, void* buf, int32_t n_seg, int64_t extra_cap);
int64_t table_build_workspace_bytes(int64_t total, int32_t n_seg, int64_t total_buckets);
// Prefix-index maintenance (k_index.hip).  One commit of a routed batch.
constexpr int64_t kSelChunk = 4096;           // candidates per selection chunk
struct IndexCommit {
    int32_t N = 0, R = 0;
    uint32_t epoch = 0;
    int n_cu = 1;
    const int64_t* req_off = nullptr;       // routed batch (device)
    const uint64_t* req_hashes = nullptr;
    const int32_t* chosen = nullptr;
    const int64_t* off = nullptr;           // current lists; stamps touched in place
    const uint64_t* hash = nullptr;
    uint64_t* stamp = nullptr;
    const uint32_t* entry_of = nullptr;     // table slot -> list entry
    const int64_t* eidx = nullptr;          // [N] entry of the all-ones key, -1 if absent
    const int64_t* capacity = nullptr;      // [N] blocks
    int64_t* occ = nullptr;                 // [N] workspace
    int64_t* fbase = nullptr;               // [N + 1] batch-local set buckets
    uint64_t* fkey = nullptr;
    uint64_t* fstamp = nullptr;
    int64_t fresh_slots_bound = 0;
    int64_t* fcount = nullptr;              // [N]
    uint64_t* efresh = nullptr;             // [N]
    int64_t* cand = nullptr;                // [N]
    int64_t* off2 = nullptr;                // [N + 1] new lists
    uint64_t* hash2 = nullptr;
    uint64_t* stamp2 = nullptr;
    // selection of each instance's survivors, in chunks of candidates
    int64_t* nvirt = nullptr;               // [N] candidate positions (listed, set slots, all-ones)
    int64_t* chunk0 = nullptr;              // [N + 1] first chunk of each instance
    int64_t chunk_bound = 0;                // upper bound of chunk0[N]
    int64_t* sel_want = nullptr;            // [N]
    uint64_t* sel_prefix = nullptr;         // [N]
    uint64_t* sel_mask = nullptr;           // [N]
    int64_t* sel_pos = nullptr;             // [N]
    int64_t* sel_active = nullptr;          // [N]
    uint32_t* sel_hist = nullptr;           // [N x 256]
};
hipError_t launch_position_stamps(const int64_t* off, int32_t N, uint64_t* stamp, int64_t total, int n_cu,
                                  hipStream_t s);
hipError_t launch_entry_map(const CacheTables& T, const int64_t* off, int32_t N, const uint64_t* hash,
                            uint32_t* entry_of, int64_t* eidx, int64_t total_bound, int n_cu, hipStream_t s);
hipError_t launch_live_entries(const CacheTables& T, const int64_t* off, int32_t N, const uint64_t* hash,
                               const uint32_t* entry_of, const int64_t* eidx, uint8_t* live, int64_t total_bound,
                               int n_cu, hipStream_t s);
hipError_t launch_dedup_lists(const int64_t* off, int32_t N, const uint64_t* hash, const uint64_t* stamp,
                              const uint8_t* live, int64_t* cand, int64_t* off2, uint64_t* hash2, uint64_t* stamp2,
                              hipStream_t s);
hipError_t launch_commit(const CacheTables& T, const IndexCommit& C, hipStream_t s);

hipError_t launch_table_build(const CacheTables& t, const int64_t* inst_off, const int32_t* seg_off, int32_t n_seg,
                              const uint64_t* hashes, int64_t total, int32_t n_inst, void* ovf_ws, int n_cu,
                              hipStream_t s, uint32_t* entry_of = nullptr,
                              int64_t* eidx = nullptr);

// Group table for the prefix-sharing pass: a power of two >= 2R slots.
inline int64_t group_table_size(int32_t R) {
    int64_t g = 64;
    while (g < 2 * (int64_t)R) g <<= 1;
    return g;
}
int64_t prefix_workspace_bytes(int32_t R, int32_t N);
// Whether followers' continuations go through the semi-join (mode 0 decides
// from the sizes, 1 always, 2 never).
bool prefix_use_join(int32_t R, int32_t N, int64_t table_slots, int mode);
// closed: leaders search the run end instead of walking it (exact only when
// every cache is prefix-closed for every prompt).
hipError_t launch_prefix_match(const CacheTables& t, int32_t R, int32_t N, const int64_t* req_off,
                               const uint64_t* req_hashes, int32_t* overlap, void* workspace, int n_cu,
                               bool join, bool closed, hipStream_t s);

hipError_t launch_refresh_compute_copy(const ModelDims& m, const float* master, float* compute, hipStream_t s);
hipError_t launch_instance_partial(const ModelDims& m, const float* compute, const float* mu,
                                   const float* inv_sigma, const float* inst_feat, int32_t N, float* part_t,
                                   hipStream_t s);
hipError_t launch_score_pairs(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                              const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                              const int32_t* prompt_len, const int32_t* overlap, float* scores, hipStream_t s);
// The same canonical scores on the matrix cores (two hidden layers of equal
// width 64, 128 or 256): bit-identical to launch_score_pairs.  With list and
// count (device; both or neither) only the pairs list[0 .. *count) are scored,
// as launch_rescore does.
bool chain_mfma_supported(const ModelDims& m);
hipError_t launch_score_chain_mfma(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                                   const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                                   const int32_t* prompt_len, const int32_t* overlap, const int64_t* list,
                                   const uint32_t* count, int n_cu, float* scores, hipStream_t s);
hipError_t launch_argmin(const ModelDims& m, int32_t R, int32_t N, const float* scores, const uint8_t* band,
                         const int64_t* req_off, const int32_t* prompt_len, const int32_t* overlap,
                         const float* inst_feat, int32_t* chosen, float* min_ttft, float* feat_out, hipStream_t s);

hipError_t launch_prepare_mfma(const MfmaLayout& L, const float* master, uint16_t* frag16, float* frag32,
                               hipStream_t s);
hipError_t launch_score_pairs_mfma(const ModelDims& m, const uint16_t* frag16, const float* frag32,
                                   const float* compute, const float* part_t, const float* mu,
                                   const float* inv_sigma, int32_t R, int32_t N, const int64_t* req_off,
                                   const int32_t* prompt_len, const int32_t* overlap, float* scores, float* errb,
                                   int n_cu, hipStream_t s);
hipError_t launch_band_select(int32_t R, int32_t N, const float* t, const float* E, uint8_t* band, int64_t* list,
                              uint32_t* count, hipStream_t s);
struct PolicyStats;
struct PolicyArgs;
// Band selection for the routing policy: delta >= 0 widens the band to every
// possible near-best pair, k_filter > 0 adds the K-filter's instances when the
// batch is saturated (stats on the device).
hipError_t launch_band_select_policy(int32_t R, int32_t N, const float* t, const float* E, double delta,
                                     int32_t k_filter, const PolicyStats* stats, const int64_t* req_off,
                                     const uint64_t* req_hashes, uint8_t* band, int64_t* list, uint32_t* count,
                                     hipStream_t s);
// Two-stage candidate selection of a scoring call: the fast argmin of each
// request first (lead[r], to be rescored), then, from its canonical score in
// `canon`, every pair that can still be the canonical argmin or near-best.
hipError_t launch_band_lead(int32_t R, int32_t N, const float* t, int64_t* lead, hipStream_t s);
hipError_t launch_band_rest(int32_t R, int32_t N, const float* t, const float* E, const float* canon,
                            const int64_t* lead, double delta, int32_t k_filter, const PolicyStats* stats,
                            const int64_t* req_off, const uint64_t* req_hashes, uint8_t* band, int64_t* list,
                            uint32_t* count, hipStream_t s);
hipError_t launch_policy_stats(const PolicyArgs& P, const float* inst_feat, int32_t N, int d_inst, double* cnt,
                               PolicyStats* st, hipStream_t s);
hipError_t launch_route(const PolicyArgs& P, const PolicyStats* st, const double* cnt, const ModelDims& m, int32_t R,
                        int32_t N, const int64_t* req_off, const uint64_t* req_hashes, const int32_t* prompt_len,
                        const int32_t* overlap, const float* scores, const uint8_t* band, const float* inst_feat,
                        const uint32_t* rnd, int32_t* chosen, int32_t* status, int32_t* heur, float* feat_out,
                        hipStream_t s);
hipError_t launch_rescore(const ModelDims& m, const float* compute, const float* mu, const float* inv_sigma,
                          const float* part_t, int32_t R, int32_t N, const int64_t* req_off,
                          const int32_t* prompt_len, const int32_t* overlap, const int64_t* list,
                          const uint32_t* count, float* scores, int n_cu, hipStream_t s);

// Forward pass of B raw rows (canonical chains, kernel precision); the last
// hidden layer's activations [hl][B] and t [B] point into ws, which holds
// forward_rows_floats(m, B) floats.
int64_t forward_rows_floats(const ModelDims& m, int32_t B);
hipError_t launch_forward_rows(const ModelDims& m, const float* compute, const float* mu, const float* isig, int32_t B,
                               const float* feats, float* ws, float** alast_out, float** t_out, hipStream_t s);
// Scores of all R x N pairs for models without two hidden layers, in chunks
// through the same forward; ws holds generic_score_floats(m, R * N) floats.
int64_t generic_score_floats(const ModelDims& m, int64_t pairs);
hipError_t launch_score_generic(const ModelDims& m, const float* compute, const float* mu, const float* isig,
                                int32_t R, int32_t N, const int64_t* req_off, const int32_t* prompt_len,
                                const int32_t* overlap, const float* inst_feat, float* scores, float* ws, int n_cu,
                                hipStream_t s);

// Online-learning data path: row gathers and scatters, and the gradient-coreset
// admission of nc candidates into a pool of n0 members (cap slots).
hipError_t launch_gather_rows(const int32_t* code, int32_t n, int d, const float* ax, const float* ay,
                              const float* bx, const float* by, float* ox, float* oy, hipStream_t s);
hipError_t launch_scatter_rows(const int32_t* dst, int32_t n, int d, const float* x, const float* y, float* fx,
                               float* fy, hipStream_t s);
// Candidates are decided in chunks of admission_chunk(nc): dcp holds
// chunk x cap distances, dcc chunk x chunk, origin cap slots, row and redo cap,
// rslots chunk + 1.
int32_t admission_chunk(int32_t nc);
hipError_t launch_admission(const float* a2, const float* t, const float* y_all, int32_t n0, int32_t nc, int H, int d,
                            int32_t cap, const float* cx, const float* cy, double* cemb, double* emb, float* rx,
                            float* ry, double* D, double* nnd, int32_t* nni, double* row, int32_t* redo,
                            int32_t* admitted, double* dcp, double* dcc, int32_t* origin, int32_t* rslots,
                            hipStream_t s);
hipError_t launch_loss_accumulate(const float* loss, double* acc, int reset, hipStream_t s);
hipError_t launch_loss_finish(const double* acc, int32_t count, float* out, hipStream_t s);

// Online update.  Workspace layout is chosen by update_workspace_floats().
int64_t update_workspace_bytes(const ModelDims& m, int32_t B);
hipError_t launch_update(const ModelDims& m, float* master, float* compute, const float* mu,
                         const float* inv_sigma, int32_t B, const float* feats, const float* ttft, float lr,
                         float* loss_out, float* grad_out, void* workspace, const DropArgs& drop, int n_cu,
                         hipStream_t s);

}  // namespace ls
