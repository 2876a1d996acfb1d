// Host side of liblodestar: the C ABI declared in include/lodestar.h.
//
// Every entry point validates its arguments on the host before enqueuing
// anything, keeps the caller's device current only for its own duration, and
// reports failures through a status code plus a per-context message.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ls_internal.h"
#include "k_policy.h"

struct ls_ctx {
    ls_model_config cfg{};
    ls::ModelDims dims;
    int device = 0;
    std::string err;
    // model (fp32 masters in the ABI packing, the kernels' compute copy, z-score stats)
    float* master = nullptr;
    float* compute = nullptr;
    float* mu = nullptr;
    float* isig = nullptr;
    bool have_model = false;
    // bf16 matrix-core path (fragment tables derived from the masters)
    uint16_t* frag16 = nullptr;
    float* frag32 = nullptr;
    bool exact_scores = false;
    // shadow model for double-buffered retraining: updates act on it, scoring
    // on the live model above, until ls_swap_model exchanges the two
    bool shadow_on = false;
    float *sh_master = nullptr, *sh_compute = nullptr, *sh_frag32 = nullptr;
    uint16_t* sh_frag16 = nullptr;
    hipEvent_t swap_ev[2] = {nullptr, nullptr};
    // dropout while training: rate, seed and the number of update calls since it was set
    double drop_p = 0.0;
    uint64_t drop_seed = 0, drop_step = 0;
    int prefix_join = 0;     // 0 decide per call, 1 always, 2 never
    bool prefix_closed = false;
    int n_cu = 1;            // compute units the launches are sized for (ls_set_cu_limit)
    int n_cu_dev = 1;        // compute units of the device
    // cache state
    ls::CacheTables tables;
    int64_t table_cap_buckets = 0;
    int32_t inst_cap = 0;
    int64_t* inst_off_dev = nullptr;
    int32_t* seg_off_dev = nullptr;    // [N + 1] first table segment of each instance
    char* inst_meta = nullptr;         // one block: tables.base, tables.nbuckets, inst_off_dev, seg_off_dev
    void* tws = nullptr;               // table-build workspace: key partition, overflow queue
    size_t tws_cap = 0;
    void* fpb = nullptr;               // fingerprints of the cached keys (tables.fp and the rest)
    size_t fpb_cap = 0;
    int64_t tables_nseg = 0;           // table segments of the loaded layout
    bool have_cache = false;
    // prefix-index maintenance: per-instance lists with recency stamps
    struct Index {
        bool on = false;                   // capacities set: loads keep the lists
        bool live = false;                 // lists of the loaded state present
        std::vector<int64_t> capacity;     // [n] blocks per instance
        int32_t n = 0;
        uint32_t epoch = 0;                // commits since the load
        int64_t list_entries = 0;          // entries each list buffer holds
        uint64_t *hash = nullptr, *stamp = nullptr, *hash2 = nullptr, *stamp2 = nullptr;
        size_t hash_cap = 0, stamp_cap = 0, hash2_cap = 0, stamp2_cap = 0;
        uint32_t* entry_of = nullptr;      // [table slots] list entry of the key in a slot
        size_t entry_cap = 0;
        int64_t* small = nullptr;          // per-instance arrays (layout in index_small)
        size_t small_cap = 0;
        int64_t *off = nullptr, *off2 = nullptr;   // [n + 1] each, inside `small`
        void* ws = nullptr;                // batch-local sets, live flags
        size_t ws_cap = 0;
    } idx;
    // grow-only workspace
    void* ws = nullptr;
    size_t ws_cap = 0;
    // scratch of ls_update alone, so that an update on a training stream never
    // shares memory with a scoring call on another stream
    void* upd_ws = nullptr;
    size_t upd_ws_cap = 0;
    // online-learning data path (device pools, host-side counters)
    struct Buffer {
        int32_t fifo_cap = 0, rep_cap = 0, fifo_count = 0, fifo_head = 0, rep_count = 0;
        float *fifo_x = nullptr, *fifo_y = nullptr, *rep_x = nullptr, *rep_y = nullptr;
        double *emb = nullptr, *nnd = nullptr, *D = nullptr;   // D: pairwise distances [rep_cap x rep_cap]
        int32_t* nni = nullptr;
        void* ws = nullptr;
        size_t ws_cap = 0;
    } buf;
    // pinned staging for host -> device copies, reusable once `stage_done` has fired
    void* stage = nullptr;
    size_t stage_cap = 0;
    hipEvent_t stage_done = nullptr;
    bool stage_pending = false;
    // optional per-kernel timing
    bool profiling = false;
    // shared_start: the start is the stop of the record before it (its
    // owner), so it is released and destroyed with that record only
    struct Rec { int kind; hipEvent_t start, stop; bool shared_start; };
    std::vector<Rec> recs;
    std::vector<hipEvent_t> spare;
    hipEvent_t last_stop = nullptr;          // stop of the group timed last, while the next may follow it
    hipStream_t last_stop_stream = nullptr;
};

// Scratch of the allocation-free scoring entry point: one array per GPU,
// reserved while the library is loaded.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in for the symbol); it uses
// the device address that hipGetSymbolAddress returns for the current device.
constexpr size_t kNoAllocScratchBytes = LS_NOALLOC_SCRATCH_BYTES;
static_assert(kNoAllocScratchBytes % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
hipError_t g_scratch_err[kMaxScratchDevices] = {};

// Device address of `scratch` on `device`, looked up once per device with that
// device current (the caller's DeviceScope); nullptr if the lookup failed.
void* scratch_on(int device) {
    if (device < 0 || device >= kMaxScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device] && g_scratch_err[device] == hipSuccess) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            g_scratch_err[device] = e != hipSuccess ? e : hipErrorInvalidSymbol;
            (void)hipGetLastError();
        } else {
            g_scratch_ptr[device] = ptr;
        }
    }
    return g_scratch_ptr[device];
}

int fail(ls_ctx* c, int code, const char* fmt, ...) {
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        c->err = buf;
    }
    return code;
}

#define LS_HIP(ctx, expr)                                                                          \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess)                                                                      \
            return fail((ctx), LS_ERR_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));       \
    } while (0)

// Makes ctx->device current for the scope and restores the caller's device.
struct DeviceScope {
    int prev = -1;
    bool ok = false;
    explicit DeviceScope(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceScope() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// The model that updates act on: the shadow while double buffering, else the live one.
struct ModelSlot {
    float* master;
    float* compute;
    uint16_t* frag16;
    float* frag32;
};
ModelSlot train_model(ls_ctx* c) {
    if (c->shadow_on) return {c->sh_master, c->sh_compute, c->sh_frag16, c->sh_frag32};
    return {c->master, c->compute, c->frag16, c->frag32};
}

// Copy one model slot onto another on stream s.
hipError_t copy_model(ls_ctx* c, const ModelSlot& to, const ModelSlot& from, hipStream_t s) {
    hipError_t e = hipMemcpyAsync(to.master, from.master, sizeof(float) * (size_t)c->dims.n_params,
                                  hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(to.compute, from.compute, sizeof(float) * (size_t)c->dims.n_compute,
                           hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && from.frag16) {
        const ls::MfmaLayout L = ls::make_mfma_layout(c->dims);
        e = hipMemcpyAsync(to.frag16, from.frag16, sizeof(uint16_t) * (size_t)L.n16, hipMemcpyDeviceToDevice, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(to.frag32, from.frag32, sizeof(float) * (size_t)L.n32, hipMemcpyDeviceToDevice, s);
    }
    return e;
}

// The dropout of the next update call (and count it).
ls::DropArgs next_drop(ls_ctx* c) {
    ls::DropArgs D;
    if (c->drop_p > 0.0) {
        D.seed = c->drop_seed;
        D.step = c->drop_step++;
        D.thr53 = (uint64_t)ldexp(c->drop_p, 53);
        D.scale = (float)(1.0 / (1.0 - c->drop_p));
    }
    return D;
}

bool valid_config(const ls_model_config* cfg, std::string* why) {
    if (!cfg) { *why = "config is NULL"; return false; }
    if (cfg->d <= LS_DERIVED_COLS || cfg->d > 4096) { *why = "d must be in (5, 4096]"; return false; }
    if (cfg->n_hidden < 1 || cfg->n_hidden > LS_MAX_HIDDEN) { *why = "n_hidden must be 1..3"; return false; }
    for (int l = 0; l < cfg->n_hidden; ++l)
        if (cfg->hidden[l] < 1 || cfg->hidden[l] > 512) { *why = "hidden widths must be 1..512"; return false; }
    if (cfg->block_tokens < 1) { *why = "block_tokens must be >= 1"; return false; }
    if (cfg->dtype != LS_FP32 && cfg->dtype != LS_BF16) { *why = "dtype must be LS_FP32 or LS_BF16"; return false; }
    return true;
}

// Wait for the last staged copy before the host buffer is rewritten; grow it if needed.
int stage_reserve(ls_ctx* c, size_t bytes) {
    if (c->stage_pending) {
        LS_HIP(c, hipEventSynchronize(c->stage_done));
        c->stage_pending = false;
    }
    if (bytes > c->stage_cap) {
        if (c->stage) LS_HIP(c, hipHostFree(c->stage));
        c->stage = nullptr;
        c->stage_cap = 0;
        size_t cap = (size_t)round_up((int64_t)bytes, 1 << 16);
        if (hipHostMalloc(&c->stage, cap, hipHostMallocDefault) != hipSuccess) {
            c->stage = nullptr;
            return fail(c, LS_ERR_NOMEM, "pinned staging allocation of %zu bytes failed", cap);
        }
        c->stage_cap = cap;
    }
    return LS_OK;
}

int stage_copy(ls_ctx* c, void* dst, size_t bytes, hipStream_t s) {
    LS_HIP(c, hipMemcpyAsync(dst, c->stage, bytes, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    return LS_OK;
}

// Grow-only device buffer, ordered on the stream of the call that needs it:
// the old buffer is released by hipFreeAsync after the work already enqueued on
// `s` (its last users), and the new one comes from the stream-ordered
// allocator, so growing never waits for the device or for other streams.
int grow(ls_ctx* c, void** p, size_t* cap, size_t bytes, hipStream_t s) {
    if (bytes <= *cap) return LS_OK;
    if (*p) {
        LS_HIP(c, hipFreeAsync(*p, s));
        *p = nullptr;
        *cap = 0;
    }
    size_t want = (size_t)round_up((int64_t)bytes, 1 << 20);
    if (hipMallocAsync(p, want, s) != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(c, LS_ERR_NOMEM, "device allocation of %zu bytes failed", want);
    }
    *cap = want;
    return LS_OK;
}

enum Kind {
    K_TABLE = 0, K_PREFIX, K_PARTIAL, K_SCORE, K_ARGMIN, K_UPDATE, K_SCORE_MFMA, K_BAND, K_RESCORE, K_ROUTE, K_BUFFER,
    K_INDEX, K_COUNT
};
const char* const kKindNames[K_COUNT] = {"table_build", "prefix_match", "instance_partial", "score_pairs", "argmin",
                                         "update", "score_pairs_mfma", "band_select", "rescore", "route",
                                         "buffer", "index"};

hipEvent_t take_event(ls_ctx* c) {
    if (!c->spare.empty()) {
        hipEvent_t e = c->spare.back();
        c->spare.pop_back();
        return e;
    }
    // timing only: without the system-scope fence a record costs no L2
    // writeback, so the events do not stretch the work they bracket
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

// Brackets one launch group with events when profiling is on.  A group that
// follows another on the same stream with nothing enqueued between them
// (`follows`) starts at the other's stop event instead of a new one: one
// event per boundary, each event record costing the stream a short idle gap.
struct Timed {
    ls_ctx* c;
    int kind;
    hipStream_t s;
    hipEvent_t start = nullptr;
    bool shared = false;
    Timed(ls_ctx* c_, int kind_, hipStream_t s_, bool follows = false) : c(c_), kind(kind_), s(s_) {
        if (!c->profiling) return;
        if (follows && c->last_stop && c->last_stop_stream == s) {
            start = c->last_stop;
            shared = true;
        } else if ((start = take_event(c)) != nullptr) {
            (void)hipEventRecord(start, s);
        }
        c->last_stop = nullptr;
    }
    void done() {
        if (!start) return;
        hipEvent_t stop = take_event(c);
        if (stop && hipEventRecord(stop, s) == hipSuccess) {
            c->recs.push_back({kind, start, stop, shared});
            c->last_stop = stop;
            c->last_stop_stream = s;
        } else {
            if (!shared) c->spare.push_back(start);
            if (stop) c->spare.push_back(stop);
        }
        start = nullptr;
    }
};

#define LS_TIMED(ctx, kind, s, expr)        \
    do {                                     \
        Timed t_((ctx), (kind), (s));        \
        hipError_t e2_ = (expr);             \
        t_.done();                           \
        LS_HIP((ctx), e2_);                  \
    } while (0)

// A group enqueued right after the timed group before it, on the same stream.
#define LS_TIMED_NEXT(ctx, kind, s, expr)    \
    do {                                     \
        Timed t_((ctx), (kind), (s), true);  \
        hipError_t e2_ = (expr);             \
        t_.done();                           \
        LS_HIP((ctx), e2_);                  \
    } while (0)

struct WsCarve {
    char* base;
    size_t cap = SIZE_MAX;   // bytes behind base
    size_t off = 0;
    template <class T>
    T* take(int64_t count) {
        T* p = reinterpret_cast<T*>(base + off);
        off += (size_t)round_up(count * (int64_t)sizeof(T), 256);
        return p;
    }
    bool ok() const { return off <= cap; }
};

}  // namespace

namespace ls {

ModelDims make_dims(const ls_model_config& cfg) {
    ModelDims m;
    m.d = cfg.d;
    m.d_inst = cfg.d - LS_DERIVED_COLS;
    m.L = cfg.n_hidden;
    for (int l = 0; l < m.L; ++l) m.h[l] = cfg.hidden[l];
    m.hl = m.h[m.L - 1];
    m.h1 = m.h[0];
    m.h2 = m.L >= 2 ? m.h[1] : 0;
    m.bf16 = cfg.dtype == LS_BF16;
    m.block_tokens = cfg.block_tokens;
    // masters: the ABI packing, per layer W [out x in] then b [out]
    int64_t o = 0;
    for (int l = 0; l <= m.L; ++l) {
        m.m_w[l] = o; o += (int64_t)m.out_of(l) * m.in_of(l);
        m.m_b[l] = o; o += m.out_of(l);
    }
    m.n_params = o;
    if (m.L == 2) {
        m.m_w1 = m.m_w[0]; m.m_b1 = m.m_b[0];
        m.m_w2 = m.m_w[1]; m.m_b2 = m.m_b[1];
        m.m_w3 = m.m_w[2]; m.m_b3 = m.m_b[2];
        // compute copy of the fused two-layer scorers
        o = 0;
        m.c_w1 = o; o += (int64_t)m.h1 * m.d;
        m.c_b1 = o; o += m.h1;
        m.c_w2t = o; o += (int64_t)m.h1 * m.h2;
        m.c_b2 = o; o += m.h2;
        m.c_w3 = o; o += m.h2;
        m.c_b3 = o; o += 1;
        m.c_w1t = o; o += (int64_t)m.d * m.h1;
        m.n_compute = o;
        m.c_wt[0] = m.c_w1t; m.c_bl[0] = m.c_b1;
        m.c_wt[1] = m.c_w2t; m.c_bl[1] = m.c_b2;
        m.c_wt[2] = m.c_w3;  m.c_bl[2] = m.c_b3;
    } else {
        // every layer transposed, W_l^T [in x out], then its bias
        o = 0;
        for (int l = 0; l <= m.L; ++l) {
            m.c_wt[l] = o; o += (int64_t)m.in_of(l) * m.out_of(l);
            m.c_bl[l] = o; o += m.out_of(l);
        }
        m.n_compute = o;
    }
    return m;
}

}  // namespace ls

extern "C" {

int64_t ls_param_count(const ls_model_config* cfg) {
    std::string why;
    if (!valid_config(cfg, &why)) return -1;
    int64_t n = 0;
    int prev = cfg->d;
    for (int l = 0; l <= cfg->n_hidden; ++l) {
        int out = l < cfg->n_hidden ? cfg->hidden[l] : 1;
        n += (int64_t)out * prev + out;
        prev = out;
    }
    return n;
}

const char* ls_last_error(const ls_ctx* ctx) {
    if (!ctx) return "context is NULL";
    return ctx->err.c_str();
}

int ls_create(const ls_model_config* cfg, int device, ls_ctx** out) {
    if (!out) return LS_ERR_INVALID;
    *out = nullptr;
    std::string why;
    if (!valid_config(cfg, &why)) return LS_ERR_INVALID;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) {
        (void)hipGetLastError();
        return LS_ERR_DEVICE;
    }
    if (device < 0 || device >= ndev) return LS_ERR_INVALID;
    ls_ctx* c = new (std::nothrow) ls_ctx();
    if (!c) return LS_ERR_NOMEM;
    c->cfg = *cfg;
    c->device = device;
    c->dims = ls::make_dims(*cfg);
    DeviceScope dev(device);
    bool ok = dev.ok;
    ok = ok && hipMalloc((void**)&c->master, sizeof(float) * c->dims.n_params) == hipSuccess;
    ok = ok && hipMalloc((void**)&c->compute, sizeof(float) * c->dims.n_compute) == hipSuccess;
    ok = ok && hipMalloc((void**)&c->mu, sizeof(float) * cfg->d) == hipSuccess;
    ok = ok && hipMalloc((void**)&c->isig, sizeof(float) * cfg->d) == hipSuccess;
    ok = ok && hipEventCreateWithFlags(&c->stage_done, hipEventDisableTiming) == hipSuccess;
    ok = ok && hipDeviceGetAttribute(&c->n_cu_dev, hipDeviceAttributeMultiprocessorCount, device) == hipSuccess;
    c->n_cu = c->n_cu_dev;
    // set-up of the allocation-free entry point: this device's address of its
    // scratch array (a failed lookup only disables that entry point)
    if (ok) (void)scratch_on(device);
    if (ok && ls::mfma_supported(c->dims)) {
        const ls::MfmaLayout L = ls::make_mfma_layout(c->dims);
        ok = hipMalloc((void**)&c->frag16, sizeof(uint16_t) * L.n16) == hipSuccess &&
             hipMalloc((void**)&c->frag32, sizeof(float) * L.n32) == hipSuccess;
    }
    if (!ok) {
        (void)hipGetLastError();
        ls_destroy(c);
        return LS_ERR_NOMEM;
    }
    *out = c;
    return LS_OK;
}

void ls_destroy(ls_ctx* c) {
    if (!c) return;
    {
        DeviceScope dev(c->device);
        (void)hipDeviceSynchronize();
        for (void* p : {(void*)c->master, (void*)c->compute, (void*)c->mu, (void*)c->isig, (void*)c->frag16,
                        (void*)c->frag32, (void*)c->tables.keys, c->fpb,
                        (void*)c->inst_meta, (void*)c->tables.flags, c->tws, c->ws, (void*)c->buf.fifo_x,
                        (void*)c->buf.fifo_y, (void*)c->buf.rep_x, (void*)c->buf.rep_y, (void*)c->buf.emb,
                        (void*)c->buf.nnd, (void*)c->buf.nni, (void*)c->buf.D, c->buf.ws, (void*)c->idx.hash,
                        (void*)c->idx.stamp, (void*)c->idx.hash2, (void*)c->idx.stamp2, (void*)c->idx.entry_of,
                        (void*)c->idx.small, c->idx.ws, (void*)c->sh_master, (void*)c->sh_compute, c->upd_ws,
                        (void*)c->sh_frag16, (void*)c->sh_frag32})
            if (p) (void)hipFree(p);
        if (c->stage) (void)hipHostFree(c->stage);
        if (c->stage_done) (void)hipEventDestroy(c->stage_done);
        for (hipEvent_t e : c->swap_ev)
            if (e) (void)hipEventDestroy(e);
        for (auto& r : c->recs) {
            if (!r.shared_start) (void)hipEventDestroy(r.start);
            (void)hipEventDestroy(r.stop);
        }
        for (hipEvent_t e : c->spare) (void)hipEventDestroy(e);
        (void)hipGetLastError();
    }
    delete c;
}

int ls_set_model(ls_ctx* c, const float* params, int64_t n_params, const float* mu, const float* inv_sigma,
                 void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!params || !mu || !inv_sigma) return fail(c, LS_ERR_INVALID, "params, mu and inv_sigma must be non-NULL");
    if (n_params != c->dims.n_params)
        return fail(c, LS_ERR_INVALID, "n_params is %lld, the model needs %lld", (long long)n_params,
                    (long long)c->dims.n_params);
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const size_t pb = sizeof(float) * (size_t)n_params, db = sizeof(float) * (size_t)c->cfg.d;
    int rc = stage_reserve(c, pb + 2 * db);
    if (rc) return rc;
    char* st = (char*)c->stage;
    memcpy(st, params, pb);
    memcpy(st + pb, mu, db);
    memcpy(st + pb + db, inv_sigma, db);
    LS_HIP(c, hipMemcpyAsync(c->master, st, pb, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipMemcpyAsync(c->mu, st + pb, db, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipMemcpyAsync(c->isig, st + pb + db, db, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    LS_HIP(c, ls::launch_refresh_compute_copy(c->dims, c->master, c->compute, s));
    if (c->frag16)
        LS_HIP(c, ls::launch_prepare_mfma(ls::make_mfma_layout(c->dims), c->master, c->frag16, c->frag32, s));
    if (c->shadow_on)
        LS_HIP(c, copy_model(c, {c->sh_master, c->sh_compute, c->sh_frag16, c->sh_frag32},
                             {c->master, c->compute, c->frag16, c->frag32}, s));
    c->have_model = true;
    return LS_OK;
}

int ls_get_model(ls_ctx* c, float* params, int64_t n_params, float* mu, float* inv_sigma) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!c->have_model) return fail(c, LS_ERR_STATE, "no model has been set");
    if (params && n_params != c->dims.n_params)
        return fail(c, LS_ERR_INVALID, "n_params is %lld, the model has %lld", (long long)n_params,
                    (long long)c->dims.n_params);
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    LS_HIP(c, hipDeviceSynchronize());
    if (params) LS_HIP(c, hipMemcpy(params, c->master, sizeof(float) * (size_t)n_params, hipMemcpyDeviceToHost));
    if (mu) LS_HIP(c, hipMemcpy(mu, c->mu, sizeof(float) * (size_t)c->cfg.d, hipMemcpyDeviceToHost));
    if (inv_sigma) LS_HIP(c, hipMemcpy(inv_sigma, c->isig, sizeof(float) * (size_t)c->cfg.d, hipMemcpyDeviceToHost));
    return LS_OK;
}

namespace {

// Per-instance arrays of the index, in one allocation of kIndexSmallPerN * N + 4 int64.
constexpr int64_t kIndexSmallPerN = 16;
struct IndexSmall {
    int64_t *off_a, *off_b, *cap, *eidx, *occ, *fbase, *fcount, *cand, *nvirt, *chunk0, *want, *pos, *active;
    uint64_t *efresh, *prefix, *mask;
};
IndexSmall index_small(int64_t* p, int32_t N) {
    IndexSmall m;
    m.off_a = p; p += N + 1;
    m.off_b = p; p += N + 1;
    m.cap = p; p += N;
    m.eidx = p; p += N;
    m.occ = p; p += N;
    m.fbase = p; p += N + 1;
    m.fcount = p; p += N;
    m.cand = p; p += N;
    m.efresh = reinterpret_cast<uint64_t*>(p); p += N;
    m.nvirt = p; p += N;
    m.chunk0 = p; p += N + 1;
    m.want = p; p += N;
    m.prefix = reinterpret_cast<uint64_t*>(p); p += N;
    m.mask = reinterpret_cast<uint64_t*>(p); p += N;
    m.pos = p; p += N;
    m.active = p;
    return m;
}

// After a load under ls_set_cache_capacity: the loaded hashes become the
// instances' lists (entry j stamped j + 1; a repeated key keeps its newest
// entry), and every table slot learns its key's list entry.
int index_load(ls_ctx* c, int32_t N, int64_t total, int64_t list_entries, const uint64_t* hashes, hipStream_t s) {
    auto& X = c->idx;
    const size_t lb = sizeof(uint64_t) * (size_t)(list_entries > 0 ? list_entries : 1);
    int rc;
    if ((rc = grow(c, (void**)&X.hash, &X.hash_cap, lb, s)) || (rc = grow(c, (void**)&X.stamp, &X.stamp_cap, lb, s)) ||
        (rc = grow(c, (void**)&X.hash2, &X.hash2_cap, lb, s)) || (rc = grow(c, (void**)&X.stamp2, &X.stamp2_cap, lb, s)))
        return rc;
    const int64_t slots = c->tables.total_buckets * ls::kBucketKeys;
    if ((rc = grow(c, (void**)&X.entry_of, &X.entry_cap, sizeof(uint32_t) * (size_t)slots, s))) return rc;
    if ((rc = grow(c, (void**)&X.small, &X.small_cap, sizeof(int64_t) * (size_t)(kIndexSmallPerN * N + 4), s)))
        return rc;
    if ((rc = grow(c, &X.ws, &X.ws_cap, (size_t)(total > 0 ? total : 1), s))) return rc;
    const size_t tw =
        (size_t)ls::table_build_workspace_bytes(list_entries, (int32_t)c->tables_nseg, c->tables.total_buckets);
    if ((rc = grow(c, &c->tws, &c->tws_cap, tw, s))) return rc;
    X.list_entries = list_entries;
    IndexSmall m = index_small(X.small, N);
    X.off = m.off_a;
    X.off2 = m.off_b;
    // capacities through the staging buffer
    rc = stage_reserve(c, sizeof(int64_t) * (size_t)N);
    if (rc) return rc;
    memcpy(c->stage, X.capacity.data(), sizeof(int64_t) * (size_t)N);
    LS_HIP(c, hipMemcpyAsync(m.cap, c->stage, sizeof(int64_t) * (size_t)N, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    Timed t(c, K_INDEX, s);
    LS_HIP(c, hipMemcpyAsync(X.off, c->inst_off_dev, sizeof(int64_t) * (size_t)(N + 1), hipMemcpyDeviceToDevice, s));
    if (total > 0)
        LS_HIP(c, hipMemcpyAsync(X.hash, hashes, sizeof(uint64_t) * (size_t)total, hipMemcpyDeviceToDevice, s));
    LS_HIP(c, ls::launch_position_stamps(X.off, N, X.stamp, total, c->n_cu, s));
    LS_HIP(c, ls::launch_fill_u32(X.entry_of, 0u, slots, s));
    LS_HIP(c, ls::launch_entry_map(c->tables, X.off, N, X.hash, X.entry_of, m.eidx, total, c->n_cu, s));
    uint8_t* live = static_cast<uint8_t*>(X.ws);
    LS_HIP(c, ls::launch_live_entries(c->tables, X.off, N, X.hash, X.entry_of, m.eidx, live, total, c->n_cu, s));
    LS_HIP(c, ls::launch_dedup_lists(X.off, N, X.hash, X.stamp, live, m.cand, X.off2, X.hash2, X.stamp2, s));
    std::swap(X.off, X.off2);
    std::swap(X.hash, X.hash2);
    std::swap(X.stamp, X.stamp2);
    std::swap(X.hash_cap, X.hash2_cap);
    std::swap(X.stamp_cap, X.stamp2_cap);
    LS_HIP(c, ls::launch_fill_u32(X.entry_of, 0u, slots, s));
    LS_HIP(c, ls::launch_entry_map(c->tables, X.off, N, X.hash, X.entry_of, m.eidx, total, c->n_cu, s));
    t.done();
    X.n = N;
    X.epoch = 0;
    X.live = true;
    return LS_OK;
}

}  // namespace

int ls_load_cache_state(ls_ctx* c, int32_t n_instances, const int64_t* inst_off, const uint64_t* hashes,
                        void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (n_instances < 1) return fail(c, LS_ERR_INVALID, "n_instances must be >= 1");
    if (!inst_off) return fail(c, LS_ERR_INVALID, "inst_off is NULL");
    if (inst_off[0] != 0) return fail(c, LS_ERR_INVALID, "inst_off[0] must be 0");
    for (int32_t i = 0; i < n_instances; ++i)
        if (inst_off[i + 1] < inst_off[i]) return fail(c, LS_ERR_INVALID, "inst_off decreases at %d", i);
    const int64_t total = inst_off[n_instances];
    if (total > 0 && !hashes) return fail(c, LS_ERR_INVALID, "hashes is NULL");
    if (total >= ((int64_t)1 << 32)) return fail(c, LS_ERR_UNSUPPORTED, "more than 2^32 - 1 cached blocks");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;

    // bucket layout: about four keys per 8-slot bucket (half load), built in
    // segments of kSegBuckets buckets
    const int N = n_instances;
    const bool keep_lists = c->idx.on && (int32_t)c->idx.capacity.size() == N;
    c->idx.live = false;
    c->have_cache = false;                 // until this load's build is queued
    std::vector<int64_t> base(N);
    std::vector<uint32_t> nb(N);
    std::vector<int32_t> seg_off(N + 1);
    int64_t nbk = 0, nseg = 0, list_entries = 0;
    for (int i = 0; i < N; ++i) {
        int64_t cnt = inst_off[i + 1] - inst_off[i];
        if (keep_lists && c->idx.capacity[i] > cnt) cnt = c->idx.capacity[i];   // room for the lists' growth
        list_entries += cnt;
        int64_t b = (cnt + 3) / 4;
        if (b < 1) b = 1;
        if (b > 0x7fffffff) return fail(c, LS_ERR_UNSUPPORTED, "instance %d caches too many blocks", i);
        base[i] = nbk;
        nb[i] = (uint32_t)b;
        nbk += b;
        seg_off[i] = (int32_t)nseg;
        nseg += (b + ls::kSegBuckets - 1) / ls::kSegBuckets;
        if (nseg > 0x7fffffff) return fail(c, LS_ERR_UNSUPPORTED, "cache state too large");
    }
    seg_off[N] = (int32_t)nseg;
    if (list_entries >= ((int64_t)1 << 32))
        return fail(c, LS_ERR_UNSUPPORTED, "capacities above 2^32 - 1 cached blocks in all");
    // device buffers
    size_t cap = (size_t)c->table_cap_buckets * ls::kBucketKeys * sizeof(uint64_t);
    int rc = grow(c, (void**)&c->tables.keys, &cap, (size_t)nbk * ls::kBucketKeys * sizeof(uint64_t), s);
    if (rc) return rc;
    c->table_cap_buckets = (int64_t)(cap / (ls::kBucketKeys * sizeof(uint64_t)));
    rc = grow(c, &c->tws, &c->tws_cap, (size_t)ls::table_build_workspace_bytes(total, (int32_t)nseg, nbk), s);
    if (rc) return rc;
    // fingerprints: the overflow list sized for the largest build of this
    // layout (the index maintenance rebuilds from lists of list_entries keys)
    const int64_t fp_extra = ls::table_overflow_capacity(list_entries > total ? list_entries : total);
    rc = grow(c, &c->fpb, &c->fpb_cap, (size_t)ls::table_fp_bytes((int32_t)nseg, fp_extra), s);
    if (rc) return rc;
    ls::carve_table_fp(c->tables, c->fpb, (int32_t)nseg, fp_extra);
    // metadata: bases, bucket counts, offsets and first segments, laid out in
    // one block (as in the pinned staging buffer) so that one copy moves them
    const size_t b_base = sizeof(int64_t) * N, b_nb = sizeof(uint32_t) * N, b_off = sizeof(int64_t) * (N + 1);
    const size_t o_off = (size_t)round_up((int64_t)(b_base + b_nb), 8), o_seg = o_off + b_off;
    const size_t b_seg = sizeof(int32_t) * (N + 1);
    if (N > c->inst_cap) {
        LS_HIP(c, hipDeviceSynchronize());
        for (void* p : {(void*)c->inst_meta, (void*)c->tables.flags})
            if (p) LS_HIP(c, hipFree(p));
        c->inst_meta = nullptr; c->tables.flags = nullptr;
        c->tables.base = nullptr; c->tables.nbuckets = nullptr; c->inst_off_dev = nullptr; c->seg_off_dev = nullptr;
        c->inst_cap = 0;
        bool ok = hipMalloc((void**)&c->inst_meta, o_seg + b_seg) == hipSuccess &&
                  hipMalloc((void**)&c->tables.flags, sizeof(uint32_t) * N) == hipSuccess;
        if (!ok) {
            (void)hipGetLastError();
            return fail(c, LS_ERR_NOMEM, "instance metadata allocation failed");
        }
        c->inst_cap = N;
    }
    // a smaller N than the allocation's packs into the front of the block
    c->tables.base = reinterpret_cast<int64_t*>(c->inst_meta);
    c->tables.nbuckets = reinterpret_cast<uint32_t*>(c->inst_meta + b_base);
    c->inst_off_dev = reinterpret_cast<int64_t*>(c->inst_meta + o_off);
    c->seg_off_dev = reinterpret_cast<int32_t*>(c->inst_meta + o_seg);
    rc = stage_reserve(c, o_seg + b_seg + 64);
    if (rc) return rc;
    char* st = (char*)c->stage;
    memcpy(st, base.data(), b_base);
    memcpy(st + b_base, nb.data(), b_nb);
    memcpy(st + o_off, inst_off, b_off);
    memcpy(st + o_seg, seg_off.data(), b_seg);
    LS_HIP(c, hipMemcpyAsync(c->inst_meta, st, o_seg + b_seg, hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    c->tables.n = N;
    c->tables.total_buckets = nbk;
    c->tables_nseg = nseg;
    // build
    {
        Timed t(c, K_TABLE, s);
        hipError_t e = ls::launch_table_build(c->tables, c->inst_off_dev, c->seg_off_dev, (int32_t)nseg, hashes, total,
                                              N, c->tws, c->n_cu, s);
        t.done();
        LS_HIP(c, e);
    }
    c->have_cache = true;
    if (keep_lists) {
        rc = index_load(c, N, total, list_entries, hashes, s);
        if (rc) return rc;
    }
    return LS_OK;
}

namespace {

// Common checks of a scoring call; 1 with *rc set when the call must return.
int check_batch(ls_ctx* c, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                const int32_t* prompt_len, const float* inst_feat, const int32_t* chosen, int* rc) {
    *rc = LS_OK;
    if (R < 0) return *rc = fail(c, LS_ERR_INVALID, "R must be >= 0"), 1;
    if (N < 1) return *rc = fail(c, LS_ERR_INVALID, "N must be >= 1"), 1;
    if (!c->have_model) return *rc = fail(c, LS_ERR_STATE, "no model has been set"), 1;
    if (!c->have_cache) return *rc = fail(c, LS_ERR_STATE, "no cache state has been loaded"), 1;
    if (N != c->tables.n)
        return *rc = fail(c, LS_ERR_STATE, "N is %d but the cache state has %d instances", N, c->tables.n), 1;
    if (R == 0) return 1;
    if (!req_off || !req_hashes || !prompt_len || !inst_feat || !chosen)
        return *rc = fail(c, LS_ERR_INVALID,
                          "req_off, req_hashes, prompt_len, inst_feat and chosen must be non-NULL"), 1;
    return 0;
}

// Workspace of the scoring pipeline.
// Whether a scoring call runs the bf16 model on the matrix cores: only when the
// caller does not ask for the score matrix, whose every entry must then be the
// canonical score (the matrix-core path keeps canonical scores for the
// candidate band alone).
bool fast_path(const ls_ctx* c, const float* scores) { return c->frag16 && !c->exact_scores && scores == nullptr; }

// Whether a scoring call takes the layer-by-layer forward (and its scratch):
// models other than two hidden layers.  The sizing below and run_pipeline both
// ask this.
bool layer_by_layer(const ls::ModelDims& m) { return m.L != 2; }

size_t pipeline_bytes(ls_ctx* c, int32_t R, int32_t N, bool have_overlap, bool have_scores, bool fast) {
    const ls::ModelDims& m = c->dims;
    const int64_t pairs = (int64_t)R * N;
    size_t need = (size_t)round_up((int64_t)m.h1 * N * 4, 256);
    need += (size_t)round_up(ls::prefix_workspace_bytes(R, N), 256);
    if (layer_by_layer(m)) need += (size_t)round_up(4 * ls::generic_score_floats(m, pairs), 256);
    if (!have_overlap) need += (size_t)round_up(pairs * 4, 256);
    if (!have_scores) need += (size_t)round_up(pairs * 4, 256);
    if (fast) {
        need += (size_t)round_up(pairs * 4, 256);                // error scales
        need += (size_t)round_up(pairs, 256);                    // candidate flags
        need += (size_t)round_up((int64_t)R * 8, 256);           // each request's fast argmin
        need += (size_t)round_up(pairs * 8, 256);                // candidate list
        need += 256;                                             // candidate counts
    }
    return need;
}

struct Scored {
    int32_t* ov = nullptr;
    float* sc = nullptr;
    const uint8_t* band = nullptr;   // candidates holding canonical scores (null: every pair)
};

// Overlaps and scores of every pair: canonical scores everywhere, or fast
// scores with the candidate band rescored canonically.  delta / k_filter /
// stats widen the band for the routing policy (delta < 0, k_filter 0: argmin
// only).
int run_pipeline(ls_ctx* c, WsCarve& w, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                 const int32_t* prompt_len, const float* inst_feat, int32_t* overlap, float* scores, bool fast,
                 double delta, int32_t k_filter, const ls::PolicyStats* stats, hipStream_t s, Scored* out) {
    const ls::ModelDims& m = c->dims;
    const int64_t pairs = (int64_t)R * N;
    float* part_t = w.take<float>((int64_t)m.h1 * N);
    char* prefix_ws = w.take<char>(ls::prefix_workspace_bytes(R, N));
    int32_t* ov = overlap ? overlap : w.take<int32_t>(pairs);
    float* sc = scores ? scores : w.take<float>(pairs);
    const char* undersized = "scoring scratch smaller than the call's carving (internal sizing error)";
    if (!w.ok()) return fail(c, LS_ERR_NOMEM, "%s", undersized);

    LS_TIMED(c, K_PREFIX, s,
             ls::launch_prefix_match(c->tables, R, N, req_off, req_hashes, ov, prefix_ws, c->n_cu,
                                     ls::prefix_use_join(R, N, c->tables.total_buckets * ls::kBucketKeys,
                                                         c->prefix_join),
                                     c->prefix_closed, s));
    const uint8_t* band = nullptr;
    if (layer_by_layer(m)) {
        // other depths: the pairs' rows through the layer-by-layer canonical forward
        float* gws = w.take<float>(ls::generic_score_floats(m, pairs));
        if (!w.ok()) return fail(c, LS_ERR_NOMEM, "%s", undersized);
        LS_TIMED(c, K_SCORE, s,
                 ls::launch_score_generic(m, c->compute, c->mu, c->isig, R, N, req_off, prompt_len, ov, inst_feat, sc,
                                          gws, c->n_cu, s));
        out->ov = ov;
        out->sc = sc;
        out->band = nullptr;
        return LS_OK;
    }
    LS_TIMED_NEXT(c, K_PARTIAL, s, ls::launch_instance_partial(m, c->compute, c->mu, c->isig, inst_feat, N, part_t, s));
    if (fast) {
        float* eb = w.take<float>(pairs);
        uint8_t* flags = w.take<uint8_t>(pairs);
        int64_t* lead = w.take<int64_t>(R);
        int64_t* list = w.take<int64_t>(pairs);
        uint32_t* count = w.take<uint32_t>(64);       // [0]: stage-1 candidates (R), [32]: stage 2
        if (!w.ok()) return fail(c, LS_ERR_NOMEM, "%s", undersized);
        LS_TIMED_NEXT(c, K_SCORE_MFMA, s,
                      ls::launch_score_pairs_mfma(m, c->frag16, c->frag32, c->compute, part_t, c->mu, c->isig, R, N,
                                                  req_off, prompt_len, ov, sc, eb, c->n_cu, s));
        // stage 1: every request's fast argmin, rescored; stage 2: what can still beat it
        const ls::FillOp fills[2] = {{count, (uint64_t)(uint32_t)R, 1, 4}, {count + 32, 0u, 1, 4}};
        auto lead_pass = [&]() {
            hipError_t e = ls::launch_fill_multi(fills, 2, s);
            return e != hipSuccess ? e : ls::launch_band_lead(R, N, sc, lead, s);
        };
        LS_TIMED_NEXT(c, K_BAND, s, lead_pass());
        LS_TIMED_NEXT(c, K_RESCORE, s,
                      ls::launch_rescore(m, c->compute, c->mu, c->isig, part_t, R, N, req_off, prompt_len, ov, lead,
                                         count, sc, c->n_cu, s));
        LS_TIMED_NEXT(c, K_BAND, s,
                      ls::launch_band_rest(R, N, sc, eb, sc, lead, delta, k_filter, stats, req_off, req_hashes, flags,
                                           list, count + 32, s));
        LS_TIMED_NEXT(c, K_RESCORE, s,
                      ls::launch_rescore(m, c->compute, c->mu, c->isig, part_t, R, N, req_off, prompt_len, ov, list,
                                         count + 32, sc, c->n_cu, s));
        band = flags;
    } else if (m.mfma_chains && ls::chain_mfma_supported(m)) {
        LS_TIMED_NEXT(c, K_SCORE, s,
                      ls::launch_score_chain_mfma(m, c->compute, c->mu, c->isig, part_t, R, N, req_off, prompt_len, ov,
                                                  nullptr, nullptr, c->n_cu, sc, s));
    } else {
        LS_TIMED_NEXT(c, K_SCORE, s,
                      ls::launch_score_pairs(m, c->compute, c->mu, c->isig, part_t, R, N, req_off, prompt_len, ov, sc,
                                             s));
    }
    out->ov = ov;
    out->sc = sc;
    out->band = band;
    return LS_OK;
}

}  // namespace

int ls_score_batch(ls_ctx* c, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                   const int32_t* prompt_len, const float* inst_feat, int32_t* chosen, float* min_ttft,
                   float* scores, int32_t* overlap, float* feat_out, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    int rc;
    if (check_batch(c, R, N, req_off, req_hashes, prompt_len, inst_feat, chosen, &rc)) return rc;
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const bool fast = fast_path(c, scores);
    rc = grow(c, &c->ws, &c->ws_cap, pipeline_bytes(c, R, N, overlap != nullptr, scores != nullptr, fast), s);
    if (rc) return rc;
    WsCarve w{(char*)c->ws, c->ws_cap};
    Scored out;
    rc = run_pipeline(c, w, R, N, req_off, req_hashes, prompt_len, inst_feat, overlap, scores, fast, -1.0, 0, nullptr,
                      s, &out);
    if (rc) return rc;
    LS_TIMED_NEXT(c, K_ARGMIN, s,
                  ls::launch_argmin(c->dims, R, N, out.sc, out.band, req_off, prompt_len, out.ov, inst_feat, chosen,
                                    min_ttft, feat_out, s));
    return LS_OK;
}

int ls_score_batch_noalloc(ls_ctx* c, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                           const int32_t* prompt_len, const float* inst_feat, int32_t* chosen, float* min_ttft,
                           float* scores, int32_t* overlap, float* feat_out, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    int rc;
    if (check_batch(c, R, N, req_off, req_hashes, prompt_len, inst_feat, chosen, &rc)) return rc;
    const bool fast = fast_path(c, scores);
    const size_t need = pipeline_bytes(c, R, N, overlap != nullptr, scores != nullptr, fast);
    if (need > kNoAllocScratchBytes)
        return fail(c, LS_ERR_INVALID,
                    "this batch needs %zu bytes of scratch; the allocation-free entry point has %zu (fewer pairs, "
                    "or pass overlap and scores buffers, or use ls_score_batch)",
                    need, kNoAllocScratchBytes);
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    void* base = scratch_on(c->device);
    if (!base) return fail(c, LS_ERR_DEVICE, "the scratch array of device %d has no device address", c->device);
    hipStream_t s = (hipStream_t)stream;
    // no profiling events here: creating one may allocate
    const bool prof = c->profiling;
    c->profiling = false;
    WsCarve w{(char*)base, kNoAllocScratchBytes};
    Scored out;
    rc = run_pipeline(c, w, R, N, req_off, req_hashes, prompt_len, inst_feat, overlap, scores, fast, -1.0, 0, nullptr,
                      s, &out);
    if (rc == LS_OK) {
        const hipError_t e = ls::launch_argmin(c->dims, R, N, out.sc, out.band, req_off, prompt_len, out.ov,
                                               inst_feat, chosen, min_ttft, feat_out, s);
        if (e != hipSuccess) rc = fail(c, LS_ERR_DEVICE, "%s", hipGetErrorString(e));
    }
    c->profiling = prof;
    return rc;
}

int ls_fast_scores(ls_ctx* c, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                   const int32_t* prompt_len, const float* inst_feat, float* t, float* err, uint8_t* band,
                   void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!c->frag16) return fail(c, LS_ERR_UNSUPPORTED, "this model is not scored on the matrix cores");
    if (R > 0 && (!t || !err)) return fail(c, LS_ERR_INVALID, "t and err must be non-NULL");
    int rc;
    // check_batch only tests `chosen` for NULL; t stands in for it
    if (check_batch(c, R, N, req_off, req_hashes, prompt_len, inst_feat, reinterpret_cast<const int32_t*>(t), &rc))
        return rc;
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const ls::ModelDims& m = c->dims;
    const int64_t pairs = (int64_t)R * N;
    size_t need = (size_t)round_up((int64_t)m.h1 * N * 4, 256) + (size_t)round_up(ls::prefix_workspace_bytes(R, N), 256) +
                  (size_t)round_up(pairs * 4, 256) + (size_t)round_up(pairs * 8, 256) + 256;
    rc = grow(c, &c->ws, &c->ws_cap, need, s);
    if (rc) return rc;
    WsCarve w{(char*)c->ws};
    float* part_t = w.take<float>((int64_t)m.h1 * N);
    char* prefix_ws = w.take<char>(ls::prefix_workspace_bytes(R, N));
    int32_t* ov = w.take<int32_t>(pairs);
    int64_t* list = w.take<int64_t>(pairs);
    uint32_t* count = w.take<uint32_t>(64);
    LS_TIMED(c, K_PREFIX, s,
             ls::launch_prefix_match(c->tables, R, N, req_off, req_hashes, ov, prefix_ws, c->n_cu,
                                     ls::prefix_use_join(R, N, c->tables.total_buckets * ls::kBucketKeys,
                                                         c->prefix_join),
                                     c->prefix_closed, s));
    LS_TIMED(c, K_PARTIAL, s, ls::launch_instance_partial(m, c->compute, c->mu, c->isig, inst_feat, N, part_t, s));
    LS_TIMED(c, K_SCORE_MFMA, s,
             ls::launch_score_pairs_mfma(m, c->frag16, c->frag32, c->compute, part_t, c->mu, c->isig, R, N, req_off,
                                         prompt_len, ov, t, err, c->n_cu, s));
    if (band) {
        LS_TIMED(c, K_BAND, s, ls::launch_fill_u32(count, 0u, 1, s));
        LS_TIMED(c, K_BAND, s, ls::launch_band_select(R, N, t, err, band, list, count, s));
    }
    return LS_OK;
}

int ls_route_batch(ls_ctx* c, const ls_policy* pol, int32_t R, int32_t N, const int64_t* req_off,
                   const uint64_t* req_hashes, const int32_t* prompt_len, const float* inst_feat, const uint32_t* rnd,
                   int32_t* chosen, int32_t* status, int32_t* heur, float* feat_out, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!pol) return fail(c, LS_ERR_INVALID, "policy is NULL");
    const ls::ModelDims& m = c->dims;
    const int d_inst = m.d_inst;
    if (pol->heuristic != LS_HEUR_PREFIX_LOAD && pol->heuristic != LS_HEUR_PREFIX_THRESHOLD)
        return fail(c, LS_ERR_INVALID, "unknown heuristic %d", pol->heuristic);
    for (int k = 0; k < 2; ++k)
        if (pol->count_cols[k] < -1 || pol->count_cols[k] >= d_inst)
            return fail(c, LS_ERR_INVALID, "count column %d is outside [-1, %d)", pol->count_cols[k], d_inst);
    if (pol->kv_col < -1 || pol->kv_col >= d_inst)
        return fail(c, LS_ERR_INVALID, "kv column %d is outside [-1, %d)", pol->kv_col, d_inst);
    if (pol->k_filter < 0 || pol->k_filter > LS_MAX_KFILTER)
        return fail(c, LS_ERR_INVALID, "k_filter must be in [0, %d]", LS_MAX_KFILTER);
    const float fp[] = {pol->theta_imbal, pol->overload_k, pol->prefix_tau, pol->epsilon, pol->tau_sat, pol->tau_ben,
                        pol->delta};
    for (float v : fp)
        if (v != v) return fail(c, LS_ERR_INVALID, "policy parameters must not be NaN");
    if (!(pol->epsilon >= 0.0f && pol->epsilon <= 1.0f)) return fail(c, LS_ERR_INVALID, "epsilon must be in [0, 1]");
    if ((pol->lo == nullptr) != (pol->hi == nullptr))
        return fail(c, LS_ERR_INVALID, "feature bounds lo and hi must both be given or both be NULL");
    if (!rnd && (pol->epsilon > 0.0f || pol->delta >= 0.0f))
        return fail(c, LS_ERR_INVALID, "rnd is required with exploration or a tie-break");
    int rc;
    if (check_batch(c, R, N, req_off, req_hashes, prompt_len, inst_feat, chosen, &rc)) return rc;
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const bool fast = fast_path(c, nullptr);
    size_t need = pipeline_bytes(c, R, N, false, false, fast);
    need += (size_t)round_up((int64_t)N * 8, 256) + 256 + (size_t)round_up((int64_t)2 * m.d * 4, 256);
    rc = grow(c, &c->ws, &c->ws_cap, need, s);
    if (rc) return rc;
    WsCarve w{(char*)c->ws, c->ws_cap};
    double* cnt = w.take<double>(N);
    ls::PolicyStats* st = w.take<ls::PolicyStats>(1);
    float* bounds = w.take<float>(2 * (int64_t)m.d);
    ls::PolicyArgs P{};
    P.heuristic = pol->heuristic;
    P.count_col0 = pol->count_cols[0];
    P.count_col1 = pol->count_cols[1];
    P.kv_col = pol->kv_col;
    P.k_filter = pol->k_filter;
    P.cold = pol->n_samples < pol->n_min ? 1 : 0;
    P.theta_imbal = pol->theta_imbal;
    P.overload_k = pol->overload_k;
    P.prefix_tau = pol->prefix_tau;
    P.tau_sat = pol->tau_sat;
    P.tau_ben = pol->tau_ben;
    P.delta = pol->delta;
    P.explore_thr = (uint64_t)floor((double)pol->epsilon * 4294967296.0);
    if (pol->lo) {
        const size_t b = sizeof(float) * (size_t)m.d;
        rc = stage_reserve(c, 2 * b + 64);
        if (rc) return rc;
        memcpy(c->stage, pol->lo, b);
        memcpy((char*)c->stage + b, pol->hi, b);
        LS_HIP(c, hipMemcpyAsync(bounds, c->stage, 2 * b, hipMemcpyHostToDevice, s));
        LS_HIP(c, hipEventRecord(c->stage_done, s));
        c->stage_pending = true;
        P.lo = bounds;
        P.hi = bounds + m.d;
    }
    LS_TIMED(c, K_ROUTE, s, ls::launch_policy_stats(P, inst_feat, N, d_inst, cnt, st, s));
    Scored out;
    rc = run_pipeline(c, w, R, N, req_off, req_hashes, prompt_len, inst_feat, nullptr, nullptr, fast, pol->delta,
                      pol->k_filter, st, s, &out);
    if (rc) return rc;
    LS_TIMED_NEXT(c, K_ROUTE, s,
                  ls::launch_route(P, st, cnt, m, R, N, req_off, req_hashes, prompt_len, out.ov, out.sc, out.band,
                                   inst_feat, rnd, chosen, status, heur, feat_out, s));
    return LS_OK;
}

int ls_set_exact_scores(ls_ctx* c, int enable) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    c->exact_scores = enable != 0;
    return LS_OK;
}

int ls_set_chain_kernels(ls_ctx* c, int mode) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (mode != 0 && mode != 1) return fail(c, LS_ERR_INVALID, "chain kernel mode must be 0 or 1");
    c->dims.mfma_chains = mode == 0;
    return LS_OK;
}

int ls_set_cu_limit(ls_ctx* c, int n) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (n < 0) return fail(c, LS_ERR_INVALID, "the compute-unit limit must be >= 0");
    c->n_cu = (n == 0 || n > c->n_cu_dev) ? c->n_cu_dev : n;
    return LS_OK;
}

int ls_set_prefix_join(ls_ctx* c, int mode) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (mode < 0 || mode > 2) return fail(c, LS_ERR_INVALID, "prefix join mode must be 0, 1 or 2");
    c->prefix_join = mode;
    return LS_OK;
}

int ls_set_prefix_closed(ls_ctx* c, int enable) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    c->prefix_closed = enable != 0;
    return LS_OK;
}

int ls_update(ls_ctx* c, int32_t B, const float* feats, const float* ttft, float lr, float* loss_out,
              float* grad_out, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (B < 1) return fail(c, LS_ERR_INVALID, "B must be >= 1");
    if (!feats || !ttft) return fail(c, LS_ERR_INVALID, "feats and ttft must be non-NULL");
    if (!std::isfinite(lr)) return fail(c, LS_ERR_INVALID, "lr must be finite");
    if (!c->have_model) return fail(c, LS_ERR_STATE, "no model has been set");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    int64_t need = ls::update_workspace_bytes(c->dims, B);
    int rc = grow(c, &c->upd_ws, &c->upd_ws_cap, (size_t)need, s);
    if (rc) return rc;
    if (c->drop_p > 0.0 && B >= (1 << 24)) return fail(c, LS_ERR_INVALID, "B must be below 2^24 with dropout");
    const ls::DropArgs D = next_drop(c);
    const ModelSlot M = train_model(c);
    // the step and the refresh of the matrix-core fragments, timed as one group
    auto step = [&]() {
        hipError_t e = ls::launch_update(c->dims, M.master, M.compute, c->mu, c->isig, B, feats, ttft, lr, loss_out,
                                         grad_out, c->upd_ws, D, c->n_cu, s);
        if (e == hipSuccess && M.frag16)
            e = ls::launch_prepare_mfma(ls::make_mfma_layout(c->dims), M.master, M.frag16, M.frag32, s);
        return e;
    };
    LS_TIMED(c, K_UPDATE, s, step());
    return LS_OK;
}

// ---------------------------------------------------------------------------
// online-learning data path
// ---------------------------------------------------------------------------
int ls_buffer_init(ls_ctx* c, int32_t fifo_cap, int32_t replay_cap) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (fifo_cap < 1 || replay_cap < 0) return fail(c, LS_ERR_INVALID, "fifo_cap must be >= 1 and replay_cap >= 0");
    if (replay_cap > LS_MAX_REPLAY)
        return fail(c, LS_ERR_UNSUPPORTED, "replay_cap above %d (the pool keeps all pairwise distances)", LS_MAX_REPLAY);
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    LS_HIP(c, hipDeviceSynchronize());
    ls_ctx::Buffer& B = c->buf;
    for (void* p : {(void*)B.fifo_x, (void*)B.fifo_y, (void*)B.rep_x, (void*)B.rep_y, (void*)B.emb, (void*)B.nnd,
                    (void*)B.nni, (void*)B.D})
        if (p) LS_HIP(c, hipFree(p));
    B.fifo_x = B.fifo_y = B.rep_x = B.rep_y = nullptr;
    B.emb = B.nnd = B.D = nullptr;
    B.nni = nullptr;
    B.fifo_cap = B.rep_cap = B.fifo_count = B.fifo_head = B.rep_count = 0;
    const int d = c->dims.d, H = c->dims.hl;
    const int32_t rc1 = replay_cap > 0 ? replay_cap : 1;
    bool ok = hipMalloc((void**)&B.fifo_x, sizeof(float) * (size_t)fifo_cap * d) == hipSuccess &&
              hipMalloc((void**)&B.fifo_y, sizeof(float) * (size_t)fifo_cap) == hipSuccess &&
              hipMalloc((void**)&B.rep_x, sizeof(float) * (size_t)rc1 * d) == hipSuccess &&
              hipMalloc((void**)&B.rep_y, sizeof(float) * (size_t)rc1) == hipSuccess &&
              hipMalloc((void**)&B.emb, sizeof(double) * (size_t)rc1 * H) == hipSuccess &&
              hipMalloc((void**)&B.nnd, sizeof(double) * (size_t)rc1) == hipSuccess &&
              hipMalloc((void**)&B.nni, sizeof(int32_t) * (size_t)rc1) == hipSuccess &&
              hipMalloc((void**)&B.D, sizeof(double) * (size_t)rc1 * rc1) == hipSuccess;
    if (!ok) {
        (void)hipGetLastError();
        return fail(c, LS_ERR_NOMEM, "training buffer allocation failed");
    }
    B.fifo_cap = fifo_cap;
    B.rep_cap = replay_cap;
    return LS_OK;
}

int ls_buffer_state(ls_ctx* c, int32_t* fifo_count, int32_t* fifo_head, int32_t* replay_count) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (fifo_count) *fifo_count = c->buf.fifo_count;
    if (fifo_head) *fifo_head = c->buf.fifo_head;
    if (replay_count) *replay_count = c->buf.rep_count;
    return LS_OK;
}

int ls_buffer_push(ls_ctx* c, int32_t B, const float* feats, const float* ttft, int32_t* admitted, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    ls_ctx::Buffer& bf = c->buf;
    if (bf.fifo_cap < 1) return fail(c, LS_ERR_STATE, "the training buffer has not been initialised");
    if (B < 0) return fail(c, LS_ERR_INVALID, "B must be >= 0");
    if (B > 0 && (!feats || !ttft)) return fail(c, LS_ERR_INVALID, "feats and ttft must be non-NULL");
    if (!c->have_model) return fail(c, LS_ERR_STATE, "no model has been set");
    if (B == 0) return LS_OK;
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const ls::ModelDims& m = c->dims;
    const int d = m.d, H = m.hl;
    // the FIFO on the host: which rows leave it (candidates, oldest first) and where the new rows land
    std::vector<int32_t> slot_src(bf.fifo_cap);       // >= 0: old slot content, < 0: new row -(b + 1)
    for (int32_t q = 0; q < bf.fifo_cap; ++q) slot_src[q] = q;
    std::vector<int32_t> cand;                          // gather codes for the candidates
    std::vector<int32_t> dst(B, -1);
    int32_t count = bf.fifo_count, head = bf.fifo_head;
    for (int32_t b = 0; b < B; ++b) {
        int32_t slot;
        if (count < bf.fifo_cap) {
            slot = (head + count) % bf.fifo_cap;
            ++count;
        } else {
            slot = head;
            const int32_t src = slot_src[slot];
            if (src < 0) dst[-src - 1] = -1;            // a new row evicted within this push
            cand.push_back(src);
            head = (head + 1) % bf.fifo_cap;
        }
        slot_src[slot] = -(b + 1);
        dst[b] = slot;
    }
    const int32_t nc = (int32_t)cand.size();
    const int32_t n0 = bf.rep_count;
    const int32_t n_all = bf.rep_cap > 0 ? n0 + nc : 0;
    // workspace
    const int64_t f_fwd = n_all > 0 ? ls::forward_rows_floats(m, n_all) : 0;
    const int64_t ch = nc > 0 ? ls::admission_chunk(nc) : 1;
    const int64_t rcap = bf.rep_cap > 0 ? bf.rep_cap : 1;
    size_t need = (size_t)round_up((int64_t)(nc + B) * 4, 256)                       // codes
                  + (size_t)round_up((int64_t)(nc > 0 ? nc : 1) * (d + 1) * 4, 256)     // candidate rows
                  + (size_t)round_up((int64_t)(n_all > 0 ? n_all : 1) * (d + 1) * 4, 256)  // forward input
                  + (size_t)round_up(f_fwd * 4, 256)
                  + (size_t)round_up((int64_t)(nc > 0 ? nc : 1) * H * 8, 256)          // candidate embeddings
                  + (size_t)round_up((int64_t)(bf.rep_cap > 0 ? bf.rep_cap : 1) * 4, 256) + 256
                  + (size_t)round_up((int64_t)(bf.rep_cap > 0 ? bf.rep_cap : 1) * 8, 256)           // distance row
                  + (size_t)round_up(ch * rcap * 8, 256) + (size_t)round_up(ch * ch * 8, 256)     // chunk distances
                  + (size_t)round_up(rcap * 4, 256)                                              // slot origins
                  + (size_t)round_up((ch + 1) * 4, 256);                                         // slots taken
    int rc = grow(c, &bf.ws, &bf.ws_cap, need, s);
    if (rc) return rc;
    WsCarve w{(char*)bf.ws};
    int32_t* codes = w.take<int32_t>(nc + B);
    float* cx = w.take<float>((int64_t)(nc > 0 ? nc : 1) * d);
    float* cy = w.take<float>(nc > 0 ? nc : 1);
    float* ax = w.take<float>((int64_t)(n_all > 0 ? n_all : 1) * d);
    float* ay = w.take<float>(n_all > 0 ? n_all : 1);
    float* fws = w.take<float>(f_fwd > 0 ? f_fwd : 1);
    double* cemb = w.take<double>((int64_t)(nc > 0 ? nc : 1) * H);
    int32_t* redo = w.take<int32_t>(bf.rep_cap > 0 ? bf.rep_cap : 1);
    int32_t* adm = w.take<int32_t>(64);
    double* drow = w.take<double>(bf.rep_cap > 0 ? bf.rep_cap : 1);
    double* dcp = w.take<double>(ch * rcap);
    double* dcc = w.take<double>(ch * ch);
    int32_t* origin = w.take<int32_t>(rcap);
    int32_t* rslots = w.take<int32_t>(ch + 1);
    // stage the codes
    rc = stage_reserve(c, sizeof(int32_t) * (size_t)(nc + B) + 64);
    if (rc) return rc;
    if (nc) memcpy(c->stage, cand.data(), sizeof(int32_t) * (size_t)nc);
    memcpy((int32_t*)c->stage + nc, dst.data(), sizeof(int32_t) * (size_t)B);
    LS_HIP(c, hipMemcpyAsync(codes, c->stage, sizeof(int32_t) * (size_t)(nc + B), hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    // candidates leave the FIFO before the new rows overwrite it
    LS_TIMED(c, K_BUFFER, s, ls::launch_gather_rows(codes, nc, d, bf.fifo_x, bf.fifo_y, feats, ttft, cx, cy, s));
    LS_TIMED(c, K_BUFFER, s, ls::launch_scatter_rows(codes + nc, B, d, feats, ttft, bf.fifo_x, bf.fifo_y, s));
    if (n_all > 0 && nc > 0) {
        // forward of the pool (slots 0..n0) followed by the candidates
        LS_HIP(c, hipMemcpyAsync(ax, bf.rep_x, sizeof(float) * (size_t)n0 * d, hipMemcpyDeviceToDevice, s));
        LS_HIP(c, hipMemcpyAsync(ay, bf.rep_y, sizeof(float) * (size_t)n0, hipMemcpyDeviceToDevice, s));
        LS_HIP(c, hipMemcpyAsync(ax + (int64_t)n0 * d, cx, sizeof(float) * (size_t)nc * d, hipMemcpyDeviceToDevice, s));
        LS_HIP(c, hipMemcpyAsync(ay + n0, cy, sizeof(float) * (size_t)nc, hipMemcpyDeviceToDevice, s));
        float *a2 = nullptr, *t = nullptr;
        LS_TIMED(c, K_BUFFER, s,
                 ls::launch_forward_rows(m, train_model(c).compute, c->mu, c->isig, n_all, ax, fws, &a2, &t, s));
        LS_TIMED(c, K_BUFFER, s,
                 ls::launch_admission(a2, t, ay, n0, nc, H, d, bf.rep_cap, cx, cy, cemb, bf.emb, bf.rep_x, bf.rep_y,
                                      bf.D, bf.nnd, bf.nni, drow, redo, admitted ? admitted : adm, dcp, dcc,
                                      origin, rslots, s));
    } else if (admitted) {
        LS_TIMED(c, K_BUFFER, s, ls::launch_fill_u32(reinterpret_cast<uint32_t*>(admitted), 0u, 1, s));
    }
    bf.fifo_count = count;
    bf.fifo_head = head;
    bf.rep_count = bf.rep_cap > 0 ? (n0 + nc < bf.rep_cap ? n0 + nc : bf.rep_cap) : 0;
    return LS_OK;
}

int ls_buffer_read(ls_ctx* c, float* fifo_x, float* fifo_y, float* replay_x, float* replay_y, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    ls_ctx::Buffer& bf = c->buf;
    if (bf.fifo_cap < 1) return fail(c, LS_ERR_STATE, "the training buffer has not been initialised");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const int d = c->dims.d;
    // the FIFO oldest first: at most two contiguous pieces of the ring
    const int32_t first = bf.fifo_count < bf.fifo_cap - bf.fifo_head ? bf.fifo_count : bf.fifo_cap - bf.fifo_head;
    if (fifo_x && bf.fifo_count) {
        LS_HIP(c, hipMemcpyAsync(fifo_x, bf.fifo_x + (int64_t)bf.fifo_head * d, sizeof(float) * (size_t)first * d,
                                 hipMemcpyDeviceToDevice, s));
        if (bf.fifo_count > first)
            LS_HIP(c, hipMemcpyAsync(fifo_x + (int64_t)first * d, bf.fifo_x,
                                     sizeof(float) * (size_t)(bf.fifo_count - first) * d, hipMemcpyDeviceToDevice, s));
    }
    if (fifo_y && bf.fifo_count) {
        LS_HIP(c, hipMemcpyAsync(fifo_y, bf.fifo_y + bf.fifo_head, sizeof(float) * (size_t)first,
                                 hipMemcpyDeviceToDevice, s));
        if (bf.fifo_count > first)
            LS_HIP(c, hipMemcpyAsync(fifo_y + first, bf.fifo_y, sizeof(float) * (size_t)(bf.fifo_count - first),
                                     hipMemcpyDeviceToDevice, s));
    }
    if (replay_x && bf.rep_count)
        LS_HIP(c, hipMemcpyAsync(replay_x, bf.rep_x, sizeof(float) * (size_t)bf.rep_count * d, hipMemcpyDeviceToDevice,
                                 s));
    if (replay_y && bf.rep_count)
        LS_HIP(c, hipMemcpyAsync(replay_y, bf.rep_y, sizeof(float) * (size_t)bf.rep_count, hipMemcpyDeviceToDevice, s));
    return LS_OK;
}

int ls_train_round(ls_ctx* c, int32_t epochs, int32_t batch, float lr, const int32_t* perm, float* loss_out,
                   void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    ls_ctx::Buffer& bf = c->buf;
    if (bf.fifo_cap < 1) return fail(c, LS_ERR_STATE, "the training buffer has not been initialised");
    if (!c->have_model) return fail(c, LS_ERR_STATE, "no model has been set");
    if (epochs < 0 || batch < 1) return fail(c, LS_ERR_INVALID, "epochs must be >= 0 and batch >= 1");
    if (!std::isfinite(lr)) return fail(c, LS_ERR_INVALID, "lr must be finite");
    const int32_t n = bf.fifo_count + bf.rep_count;
    if (n < 1) return fail(c, LS_ERR_STATE, "the training buffer is empty");
    if (epochs == 0) return LS_OK;
    // sample k of the round: FIFO oldest first, then the pool by slot; codes for gather_rows
    std::vector<int32_t> codes((size_t)epochs * n);
    std::vector<char> seen(n);
    for (int32_t e = 0; e < epochs; ++e) {
        std::fill(seen.begin(), seen.end(), 0);
        for (int32_t k = 0; k < n; ++k) {
            const int32_t v = perm ? perm[(int64_t)e * n + k] : k;
            if (v < 0 || v >= n || seen[v]) return fail(c, LS_ERR_INVALID, "perm row %d is not a permutation of %d", e, n);
            seen[v] = 1;
            codes[(size_t)e * n + k] =
                v < bf.fifo_count ? (bf.fifo_head + v) % bf.fifo_cap : -(v - bf.fifo_count) - 1;
        }
    }
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const ls::ModelDims& m = c->dims;
    const int d = m.d;
    size_t need = (size_t)round_up((int64_t)epochs * n * 4, 256) + (size_t)round_up((int64_t)batch * (d + 1) * 4, 256) +
                  512 + (size_t)round_up(ls::update_workspace_bytes(m, batch), 256);
    int rc = grow(c, &bf.ws, &bf.ws_cap, need, s);
    if (rc) return rc;
    WsCarve w{(char*)bf.ws};
    int32_t* dcodes = w.take<int32_t>((int64_t)epochs * n);
    float* bx = w.take<float>((int64_t)batch * d);
    float* by = w.take<float>(batch);
    float* step_loss = w.take<float>(64);
    double* acc = w.take<double>(32);
    void* uws = w.take<char>(ls::update_workspace_bytes(m, batch));
    rc = stage_reserve(c, sizeof(int32_t) * codes.size() + 64);
    if (rc) return rc;
    memcpy(c->stage, codes.data(), sizeof(int32_t) * codes.size());
    LS_HIP(c, hipMemcpyAsync(dcodes, c->stage, sizeof(int32_t) * codes.size(), hipMemcpyHostToDevice, s));
    LS_HIP(c, hipEventRecord(c->stage_done, s));
    c->stage_pending = true;
    const ModelSlot TM = train_model(c);
    int32_t nb = 0;
    for (int32_t e = 0; e < epochs; ++e) {
        nb = 0;
        for (int32_t st = 0; st < n; st += batch) {
            const int32_t mb = n - st < batch ? n - st : batch;
            LS_TIMED(c, K_UPDATE, s,
                     ls::launch_gather_rows(dcodes + (int64_t)e * n + st, mb, d, bf.fifo_x, bf.fifo_y, bf.rep_x,
                                            bf.rep_y, bx, by, s));
            const ls::DropArgs D = next_drop(c);
            LS_TIMED(c, K_UPDATE, s,
                     ls::launch_update(m, TM.master, TM.compute, c->mu, c->isig, mb, bx, by, lr, step_loss, nullptr,
                                       uws, D, c->n_cu, s));
            if (e + 1 == epochs && loss_out) LS_HIP(c, ls::launch_loss_accumulate(step_loss, acc, nb == 0, s));
            ++nb;
        }
    }
    if (loss_out) LS_HIP(c, ls::launch_loss_finish(acc, nb, loss_out, s));
    if (TM.frag16)
        LS_TIMED(c, K_UPDATE, s,
                 ls::launch_prepare_mfma(ls::make_mfma_layout(c->dims), TM.master, TM.frag16, TM.frag32, s));
    return LS_OK;
}

int ls_profile_enable(ls_ctx* c, int enable) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    DeviceScope dev(c->device);
    if (!c->recs.empty()) {
        LS_HIP(c, hipDeviceSynchronize());
        for (auto& r : c->recs) {
            if (!r.shared_start) c->spare.push_back(r.start);
            c->spare.push_back(r.stop);
        }
        c->recs.clear();
    }
    c->last_stop = nullptr;
    c->profiling = enable != 0;
    return LS_OK;
}

int ls_profile_read(ls_ctx* c, int32_t max_kinds, const char** names, int64_t* launches, double* total_ms,
                    int32_t* n_kinds) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (max_kinds < 0 || (max_kinds > 0 && (!names || !launches || !total_ms)))
        return fail(c, LS_ERR_INVALID, "output arrays must hold max_kinds entries");
    DeviceScope dev(c->device);
    int64_t cnt[K_COUNT] = {};
    double ms[K_COUNT] = {};
    for (auto& r : c->recs) {
        LS_HIP(c, hipEventSynchronize(r.stop));
        float t = 0.0f;
        LS_HIP(c, hipEventElapsedTime(&t, r.start, r.stop));
        cnt[r.kind] += 1;
        ms[r.kind] += t;
    }
    int32_t k = 0;
    for (int kind = 0; kind < K_COUNT; ++kind) {
        if (!cnt[kind]) continue;
        if (k < max_kinds) {
            names[k] = kKindNames[kind];
            launches[k] = cnt[kind];
            total_ms[k] = ms[kind];
        }
        ++k;
    }
    if (n_kinds) *n_kinds = k;
    return LS_OK;
}


int ls_set_cache_capacity(ls_ctx* c, int32_t n_instances, const int64_t* capacity) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!capacity) {
        c->idx.on = false;
        c->idx.live = false;
        c->idx.capacity.clear();
        return LS_OK;
    }
    if (n_instances < 1) return fail(c, LS_ERR_INVALID, "n_instances must be >= 1");
    for (int32_t i = 0; i < n_instances; ++i)
        if (capacity[i] < 0) return fail(c, LS_ERR_INVALID, "capacity[%d] is negative", i);
    c->idx.capacity.assign(capacity, capacity + n_instances);
    c->idx.on = true;
    c->idx.live = false;                     // the lists come with the next load
    return LS_OK;
}

int ls_commit_routes(ls_ctx* c, int32_t R, int64_t n_hashes, const int64_t* req_off, const uint64_t* req_hashes,
                     const int32_t* chosen, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    auto& X = c->idx;
    if (!X.live) return fail(c, LS_ERR_STATE, "no cache state was loaded under ls_set_cache_capacity");
    if (R < 0 || R > (1 << 24)) return fail(c, LS_ERR_INVALID, "R must be in [0, 2^24]");
    if (n_hashes < 0) return fail(c, LS_ERR_INVALID, "n_hashes must be >= 0");
    if (R > 0 && (!req_off || !chosen || (n_hashes > 0 && !req_hashes)))
        return fail(c, LS_ERR_INVALID, "req_off, req_hashes and chosen must be non-NULL");
    if (X.epoch + 1 >= (1u << 20)) return fail(c, LS_ERR_STATE, "2^20 - 1 commits since the load: reload the state");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const int32_t N = X.n;
    // batch-local sets: at most n_hashes / 4 + N + 1 buckets of 8 keys and 8
    // stamps; then the selection histograms [N x 256]
    const int64_t fslots = (n_hashes / 4 + N + 1) * ls::kBucketKeys;
    int rc = grow(c, &X.ws, &X.ws_cap, sizeof(uint64_t) * 2 * (size_t)fslots + sizeof(uint32_t) * 256 * (size_t)N, s);
    if (rc) return rc;
    IndexSmall m = index_small(X.small, N);
    ls::IndexCommit C;
    C.N = N;
    C.R = R;
    C.epoch = X.epoch + 1;
    C.n_cu = c->n_cu;
    C.req_off = req_off;
    C.req_hashes = req_hashes;
    C.chosen = chosen;
    C.off = X.off;
    C.hash = X.hash;
    C.stamp = X.stamp;
    C.entry_of = X.entry_of;
    C.eidx = m.eidx;
    C.capacity = m.cap;
    C.occ = m.occ;
    C.fbase = m.fbase;
    C.fkey = static_cast<uint64_t*>(X.ws);
    C.fstamp = C.fkey + fslots;
    C.fresh_slots_bound = fslots;
    C.fcount = m.fcount;
    C.efresh = m.efresh;
    C.cand = m.cand;
    C.off2 = X.off2;
    C.hash2 = X.hash2;
    C.stamp2 = X.stamp2;
    C.nvirt = m.nvirt;
    C.chunk0 = m.chunk0;
    // chunks: sum_i ceil(nvirt_i / chunk) <= (listed + set slots + N) / chunk + N
    C.chunk_bound = (X.list_entries + fslots + N) / ls::kSelChunk + N + 1;
    C.sel_want = m.want;
    C.sel_prefix = m.prefix;
    C.sel_mask = m.mask;
    C.sel_pos = m.pos;
    C.sel_active = m.active;
    C.sel_hist = reinterpret_cast<uint32_t*>(C.fstamp + fslots);
    {
        Timed t(c, K_INDEX, s);
        LS_HIP(c, ls::launch_commit(c->tables, C, s));
        t.done();
    }
    {
        // the new lists hold each key once per instance, so the build itself
        // records every slot's list entry and the all-ones key's entry
        Timed t(c, K_TABLE, s);
        LS_HIP(c, ls::launch_fill_u64(reinterpret_cast<uint64_t*>(m.eidx), ~0ull, N, s));
        LS_HIP(c, ls::launch_table_build(c->tables, X.off2, c->seg_off_dev, (int32_t)c->tables_nseg, X.hash2,
                                         X.list_entries, N, c->tws, c->n_cu, s, X.entry_of, m.eidx));
        t.done();
    }
    std::swap(X.off, X.off2);
    std::swap(X.hash, X.hash2);
    std::swap(X.stamp, X.stamp2);
    std::swap(X.hash_cap, X.hash2_cap);
    std::swap(X.stamp_cap, X.stamp2_cap);
    X.epoch += 1;
    return LS_OK;
}

int ls_read_cache_state(ls_ctx* c, int32_t n_instances, int64_t* inst_off, uint64_t* hashes, uint64_t* stamps,
                        int64_t max_entries, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    auto& X = c->idx;
    if (!X.live) return fail(c, LS_ERR_STATE, "no cache state was loaded under ls_set_cache_capacity");
    if (n_instances != X.n) return fail(c, LS_ERR_INVALID, "n_instances is %d, the state has %d", n_instances, X.n);
    if (!inst_off) return fail(c, LS_ERR_INVALID, "inst_off is NULL");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t s = (hipStream_t)stream;
    const size_t ob = sizeof(int64_t) * (size_t)(X.n + 1);
    int rc = stage_reserve(c, ob);
    if (rc) return rc;
    LS_HIP(c, hipMemcpyAsync(c->stage, X.off, ob, hipMemcpyDeviceToHost, s));
    LS_HIP(c, hipStreamSynchronize(s));
    memcpy(inst_off, c->stage, ob);
    const int64_t total = inst_off[X.n];
    if ((hashes || stamps) && max_entries < total)
        return fail(c, LS_ERR_INVALID, "max_entries is %lld, the lists hold %lld", (long long)max_entries,
                    (long long)total);
    if (hashes && total > 0)
        LS_HIP(c, hipMemcpyAsync(hashes, X.hash, sizeof(uint64_t) * (size_t)total, hipMemcpyDeviceToDevice, s));
    if (stamps && total > 0)
        LS_HIP(c, hipMemcpyAsync(stamps, X.stamp, sizeof(uint64_t) * (size_t)total, hipMemcpyDeviceToDevice, s));
    LS_HIP(c, hipStreamSynchronize(s));
    return LS_OK;
}

int ls_set_dropout(ls_ctx* c, float p, uint64_t seed) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!(p >= 0.0f && p < 1.0f)) return fail(c, LS_ERR_INVALID, "dropout rate must be in [0, 1)");
    for (int l = 0; l < c->dims.L; ++l)
        if (c->dims.h[l] > 1024) return fail(c, LS_ERR_UNSUPPORTED, "dropout needs hidden widths up to 1024");
    c->drop_p = (double)p;
    c->drop_seed = seed;
    c->drop_step = 0;
    return LS_OK;
}

int ls_set_shadow_training(ls_ctx* c, int enable, void* stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!enable) {
        c->shadow_on = false;
        return LS_OK;
    }
    if (!c->have_model) return fail(c, LS_ERR_STATE, "no model has been set");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    if (!c->sh_master) {
        bool ok = hipMalloc((void**)&c->sh_master, sizeof(float) * c->dims.n_params) == hipSuccess &&
                  hipMalloc((void**)&c->sh_compute, sizeof(float) * c->dims.n_compute) == hipSuccess;
        if (ok && c->frag16) {
            const ls::MfmaLayout L = ls::make_mfma_layout(c->dims);
            ok = hipMalloc((void**)&c->sh_frag16, sizeof(uint16_t) * L.n16) == hipSuccess &&
                 hipMalloc((void**)&c->sh_frag32, sizeof(float) * L.n32) == hipSuccess;
        }
        ok = ok && hipEventCreateWithFlags(&c->swap_ev[0], hipEventDisableTiming) == hipSuccess &&
             hipEventCreateWithFlags(&c->swap_ev[1], hipEventDisableTiming) == hipSuccess;
        if (!ok) {
            (void)hipGetLastError();
            return fail(c, LS_ERR_NOMEM, "shadow model allocation failed");
        }
    }
    LS_HIP(c, copy_model(c, {c->sh_master, c->sh_compute, c->sh_frag16, c->sh_frag32},
                         {c->master, c->compute, c->frag16, c->frag32}, (hipStream_t)stream));
    c->shadow_on = true;
    return LS_OK;
}

int ls_swap_model(ls_ctx* c, void* serve_stream, void* train_stream) {
    if (!c) return LS_ERR_INVALID;
    c->err.clear();
    if (!c->shadow_on) return fail(c, LS_ERR_STATE, "no shadow model (ls_set_shadow_training)");
    DeviceScope dev(c->device);
    if (!dev.ok) return fail(c, LS_ERR_DEVICE, "cannot select device %d", c->device);
    hipStream_t serve = (hipStream_t)serve_stream, train = (hipStream_t)train_stream;
    // serving from here on waits for the training enqueued so far ...
    LS_HIP(c, hipEventRecord(c->swap_ev[0], train));
    LS_HIP(c, hipStreamWaitEvent(serve, c->swap_ev[0], 0));
    // ... and the old live model is overwritten only after the serving enqueued so far
    LS_HIP(c, hipEventRecord(c->swap_ev[1], serve));
    LS_HIP(c, hipStreamWaitEvent(train, c->swap_ev[1], 0));
    std::swap(c->master, c->sh_master);
    std::swap(c->compute, c->sh_compute);
    std::swap(c->frag16, c->sh_frag16);
    std::swap(c->frag32, c->sh_frag32);
    LS_HIP(c, copy_model(c, {c->sh_master, c->sh_compute, c->sh_frag16, c->sh_frag32},
                         {c->master, c->compute, c->frag16, c->frag32}, train));
    return LS_OK;
}

}  // extern "C"
