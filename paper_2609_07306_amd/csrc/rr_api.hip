// Host side of the C ABI declared in include/routerelay.h: configuration
// checks, the ledger's device allocations, and stream-ordered launches of the
// route (GEMM + TopK) and rescoring kernels.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "routerelay.h"
#include "rr_internal.hpp"
#include "rr_rescore.hpp"

struct rr_ledger {
    rr_config cfg;
    int device;
    bool has_state;
    int32_t last_layer;
    int64_t rows;
    int32_t *routes, *sent, *build, *age, *stat_nrr;
    uint8_t *flags;
    float *alpha, *beta;
    float *seed_bound, *seed_rmax;  // dense rescoring -> reroute: per-row threshold seeds (or null)
    bool fused;                     // relay layers as one pass (else rescoring + compacted reroute)
    int32_t bm_words;               // fused: ledger bitmap row stride in (R, C) word pairs
    uint32_t *done;                 // fused: finished-workgroup counter of the relay pass
    int64_t *blk_pairs;  // rescoring workgroup partials, consumed by the reroute kernel
    int32_t *blk_count;
    int64_t *stat_pairs;
};

// Device-resident library state, one copy per GPU: the running count of rows
// whose selection stopped at the collection-sweep cap, and the scratch area of
// rr_relay_layer_static (relay flags, alpha / beta, per-workgroup partials,
// call totals, threshold seeds, the one-pass completion counter).  Each GPU
// the library runs on holds its own copy until the process ends.
constexpr size_t kScratchBytes = (size_t)4 << 20;
static __device__ unsigned long long g_unconverged_dev;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_err;

constexpr int kMaxDevices = 64;

// Per-device addresses of the device-resident state, resolved with
// hipGetSymbolAddress once per device (with that device current): in host
// code the variable's name is a host-side stand-in, not a device address.
struct DeviceState {
    std::atomic<bool> ready{false};
    unsigned long long *unconverged = nullptr;
    unsigned char *scratch = nullptr;
};
DeviceState g_devstate[kMaxDevices];
std::mutex g_devstate_mu;

// Collection sweeps allowed per route tile (0: the kernel's default cap);
// lowered only by the test hook rr_set_sweep_cap.
std::atomic<int> g_sweep_cap{0};

// Diagnostics: the flagged rows of each head as an ascending id list
// (ballot + prefix over the head's flags), -1 after the last.  One
// workgroup per head.
constexpr int kIdsThreads = 256;
__global__ __launch_bounds__(kIdsThreads) void flagged_ids_kernel(const uint8_t *flags, int n_q, int32_t *ids)
{
    __shared__ int s_wave[kIdsThreads / 64];
    const uint8_t *f = flags + (int64_t)blockIdx.x * n_q;
    int32_t *o = ids + (int64_t)blockIdx.x * n_q;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int base = 0;
    for (int i0 = 0; i0 < n_q; i0 += kIdsThreads) {
        const int i = i0 + (int)threadIdx.x;
        const bool fl = i < n_q && f[i] != 0;
        const uint64_t mk = __ballot(fl);
        if (lane == 0) s_wave[w] = __popcll(mk);
        __syncthreads();
        int pre = base, tot = 0;
        for (int v = 0; v < kIdsThreads / 64; ++v) {
            pre += (v < w) ? s_wave[v] : 0;
            tot += s_wave[v];
        }
        if (fl) o[pre + __popcll(mk & ((1ull << lane) - 1ull))] = i;
        base += tot;
        __syncthreads();
    }
    for (int j = base + (int)threadIdx.x; j < n_q; j += kIdsThreads) o[j] = -1;
}

// Zeroes n 32-bit words (one small launch).
__global__ void clear_words_kernel(uint32_t *p, int n)
{
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

rr_status fail(rr_status s, const std::string &msg)
{
    g_err = msg;
    return s;
}

rr_status hip_fail(hipError_t e, const char *what)
{
    return fail(RR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

int64_t rows_of(const rr_config &c) { return (int64_t)c.n_heads * c.n_q; }

// Sentinel slots per ledger row: near-miss, random, then mandatory.
int sent_width(const rr_config &c) { return c.m + c.r + c.n_sink + c.n_recent; }

// Sum of n_i over all rows: the score pairs of one full routing pass.
int64_t full_pairs(const rr_config &c)
{
    if (!c.causal) return rows_of(c) * c.n_k;
    int64_t per_head = 0;
    for (int64_t i = 0; i < c.n_q; ++i) per_head += (i + 1 < c.n_k) ? i + 1 : c.n_k;
    return per_head * c.n_heads;
}

// Ledger bitmap row stride of the one-pass relay in (R, C) word pairs: two
// per 64 keys of the padded key range, plus one so that rows lie an odd
// number of pairs apart.
int relay_bm_words(int n_k) { return 2 * ((n_k + 63) / 64) + 1; }

rr_status validate(const rr_config *c, bool ledger)
{
    if (!c) return fail(RR_ERR_INVALID, "config is NULL");
    if ((c->options & ~(uint32_t)(RR_OPT_SPLIT_RELAY | RR_OPT_ONE_PASS_RELAY)) != 0)
        return fail(RR_ERR_INVALID, "unknown config.options bits");
    if ((c->options & RR_OPT_SPLIT_RELAY) && (c->options & RR_OPT_ONE_PASS_RELAY))
        return fail(RR_ERR_INVALID, "RR_OPT_SPLIT_RELAY and RR_OPT_ONE_PASS_RELAY exclude each other");
    if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads != 0)
        return fail(RR_ERR_INVALID, "n_heads must be a positive multiple of n_kv_heads");
    if (c->n_q < 1 || c->n_k < 1) return fail(RR_ERR_INVALID, "n_q and n_k must be >= 1");
    if (c->causal != 0 && c->causal != 1) return fail(RR_ERR_INVALID, "causal must be 0 or 1");
    if (c->causal && c->n_q != c->n_k) return fail(RR_ERR_INVALID, "the causal chunk mask needs n_q == n_k");
    if (c->dtype != RR_F32 && c->dtype != RR_BF16) return fail(RR_ERR_INVALID, "dtype must be RR_F32 or RR_BF16");
    if (c->d < 1) return fail(RR_ERR_INVALID, "d must be >= 1");
    if (c->k < 1 || c->k > c->n_k) return fail(RR_ERR_INVALID, "k must lie in [1, n_k]");
    if (c->m < 0 || c->r < 0) return fail(RR_ERR_INVALID, "m and r must be >= 0");
    if (c->n_sink < 0 || c->n_recent < 0 || c->min_reuse < 0)
        return fail(RR_ERR_INVALID, "n_sink, n_recent and min_reuse must be >= 0");
    if (c->reserved != 0) return fail(RR_ERR_INVALID, "rr_config.reserved must be 0");
    uint32_t gbits;
    std::memcpy(&gbits, &c->gamma, sizeof(gbits));
    if ((gbits & 0x7FFFFFFFu) > 0x7F800000u) return fail(RR_ERR_INVALID, "gamma is NaN");  // (bit test: device passes assume no NaN)
    const int m = ledger ? c->m : 0, r = ledger ? c->r + c->n_sink + c->n_recent : 0;
    if (!rr::route_supported(c->dtype, c->d, c->k + m))
        return fail(RR_ERR_UNSUPPORTED, "unsupported (dtype, d, k+m): d in {32,64,128} (256 for bf16), k+m <= 128");
    if (c->k + m + r > 256) return fail(RR_ERR_UNSUPPORTED, "k + m + r + n_sink + n_recent must be <= 256");
    if (c->n_k > 8192) return fail(RR_ERR_UNSUPPORTED, "n_k must be <= 8192");
    if (c->n_heads > 1024) return fail(RR_ERR_UNSUPPORTED, "n_heads must be <= 1024");
    if (rows_of(*c) * (int64_t)(c->k + m + r + 1) >= (int64_t)INT32_MAX || rows_of(*c) * c->d >= (int64_t)INT32_MAX * 8)
        return fail(RR_ERR_UNSUPPORTED, "problem too large for 32-bit row indexing");
    if (ledger && (c->options & RR_OPT_ONE_PASS_RELAY) &&
        relay_bm_words(c->n_k) > rr::route_relay_max_bm_words(c->dtype, c->d, c->k + c->m))
        return fail(RR_ERR_UNSUPPORTED, "one-pass relay: the ledger bitmaps of a tile exceed its LDS (n_k too large)");
    return RR_OK;
}

// Makes the ledger's device current for the lifetime of the guard.
struct DeviceGuard {
    int prev = -1;
    bool changed = false;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) changed = (hipSetDevice(dev) == hipSuccess);
    }
    ~DeviceGuard()
    {
        if (changed) (void)hipSetDevice(prev);
    }
};

template <typename T>
rr_status alloc(T **p, int64_t n, const char *what)
{
    *p = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(p), (size_t)(n > 0 ? n : 1) * sizeof(T));
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(RR_ERR_OOM, std::string("hipMalloc failed for ") + what);
    }
    return RR_OK;
}

void free_all(rr_ledger *L)
{
    void *ptrs[] = {L->routes, L->sent,  L->build,     L->age,       L->done,      L->stat_nrr,
                    L->flags,  L->alpha, L->beta,      L->blk_pairs, L->blk_count, L->stat_pairs,
                    L->seed_bound, L->seed_rmax};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
}

// ------------------------------------------------------------ profiling

struct ProfRecord {
    int kind;
    hipEvent_t start, stop;
};

struct Profiler {
    bool on = false;
    std::vector<ProfRecord> records;
    std::vector<hipEvent_t> pool;

    hipEvent_t get()
    {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
};

Profiler g_prof;

// Launches `fn` on `stream`, bracketed by events when profiling is on.
template <typename F>
hipError_t timed(int kind, hipStream_t stream, F fn)
{
    if (!g_prof.on) return fn();
    ProfRecord rec{kind, g_prof.get(), g_prof.get()};
    if (!rec.start || !rec.stop) return fn();
    hipError_t e = hipEventRecord(rec.start, stream);
    if (e != hipSuccess) return e;
    e = fn();
    if (e != hipSuccess) return e;
    e = hipEventRecord(rec.stop, stream);
    if (e == hipSuccess) g_prof.records.push_back(rec);
    return e;
}

// The current device's state (resolving its addresses on first use), or an
// error status with the message set.
rr_status device_state(DeviceState **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(RR_ERR_UNSUPPORTED, "device ordinal beyond the library's table");
    DeviceState &st = g_devstate[dev];
    if (!st.ready.load(std::memory_order_acquire)) {
        std::lock_guard<std::mutex> lock(g_devstate_mu);
        if (!st.ready.load(std::memory_order_relaxed)) {
            void *p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_unconverged_dev));
            if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (unconverged-row counter)");
            st.unconverged = static_cast<unsigned long long *>(p);
            p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (relay scratch)");
            st.scratch = static_cast<unsigned char *>(p);
            st.ready.store(true, std::memory_order_release);
        }
    }
    *out = &st;
    return RR_OK;
}

rr::RouteArgs route_args(const rr_config &c, const void *Q, const void *K)
{
    rr::RouteArgs a;
    std::memset(&a, 0, sizeof(a));
    a.sweep_cap = g_sweep_cap.load(std::memory_order_relaxed);
    a.Q = Q;
    a.K = K;
    a.n_heads = c.n_heads;
    a.n_kv_heads = c.n_kv_heads;
    a.n_q = c.n_q;
    a.n_k = c.n_k;
    a.d = c.d;
    a.k = c.k;
    a.m = c.m;
    a.r = c.r;
    a.n_sink = c.n_sink;
    a.n_recent = c.n_recent;
    a.min_reuse = c.min_reuse;
    a.gamma_rows = c.gamma_rows;
    a.k_rows = c.k_rows;
    a.causal = c.causal;
    a.tile_rows = rr::route_tile_rows(c.k + c.m, c.n_heads, c.n_q);
    a.tiles_per_head = (c.n_q + a.tile_rows - 1) / a.tile_rows;
    a.seed = c.seed;
    return a;
}

// Schedule of a relay layer for a configuration: by default one pass for
// causal inputs where a tile's ledger bitmaps fit its LDS (compaction would
// mix short and long causal rows in one tile), else the split schedule,
// measured faster for non-causal inputs with dense or gathered rescoring;
// and, for the split schedule with dense rescoring, whether the rescoring
// pass leaves threshold seeds.
struct RelayPlan {
    bool fused, seeds;
    int bm_words;
    rr::RescoreGeometry geo;
};

RelayPlan relay_plan(const rr_config &c)
{
    RelayPlan p;
    p.bm_words = relay_bm_words(c.n_k);
    const bool fits = p.bm_words <= rr::route_relay_max_bm_words(c.dtype, c.d, c.k + c.m);
    rr::rescore_geometry(rows_of(c), c.n_q, c.n_k, p.geo);
    p.fused = fits && ((c.options & RR_OPT_ONE_PASS_RELAY) || (!(c.options & RR_OPT_SPLIT_RELAY) && c.causal));
    p.seeds = !p.fused && p.geo.dense && rr::rescore_dense_seeds(c.dtype, c.d);
    return p;
}

// Per-workgroup partial slots a relay layer needs: one per rescoring
// workgroup (split) or per route tile (one pass).
int64_t relay_partial_slots(const rr_config &c)
{
    const int64_t rescore = (int64_t)c.n_heads * ((c.n_q + rr::kRescoreWaves - 1) / rr::kRescoreWaves);
    const int tile = rr::route_tile_rows(c.k + c.m, c.n_heads, c.n_q);
    const int64_t tiles = (int64_t)c.n_heads * ((c.n_q + tile - 1) / tile);
    return rescore > tiles ? rescore : tiles;
}

// Byte offsets of the relay scratch inside the static area (each 256-byte
// aligned) and the bytes it takes.
struct StaticLayout {
    size_t done, stat_pairs, stat_nrr, blk_pairs, blk_count, flags, alpha, beta, seed_bound, seed_rmax, bytes;
};

StaticLayout static_layout(const rr_config &c, const RelayPlan &p)
{
    const size_t rows = (size_t)rows_of(c), slots = (size_t)relay_partial_slots(c);
    StaticLayout l;
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t o = at;
        at = (at + bytes + 255) & ~(size_t)255;
        return o;
    };
    l.done = take(sizeof(uint32_t));
    l.stat_pairs = take(sizeof(int64_t));
    l.stat_nrr = take(sizeof(int32_t));
    l.blk_pairs = take(slots * sizeof(int64_t));
    l.blk_count = take(slots * sizeof(int32_t));
    l.flags = take(rows);
    l.alpha = take(rows * sizeof(float));
    l.beta = take(rows * sizeof(float));
    l.seed_bound = p.seeds ? take(rows * sizeof(float)) : 0;
    l.seed_rmax = p.seeds ? take(rows * sizeof(float)) : 0;
    l.bytes = at;
    return l;
}

// Device buffers of one relay layer: the ledger and the relay scratch.
struct RelayBuffers {
    int32_t *routes = nullptr, *sent = nullptr, *build = nullptr, *age = nullptr;
    uint8_t *flags = nullptr;
    float *alpha = nullptr, *beta = nullptr;
    float *seed_bound = nullptr, *seed_rmax = nullptr;  // split + dense rescoring: threshold seeds (or null)
    int64_t *blk_pairs = nullptr;                       // per-workgroup partials
    int32_t *blk_count = nullptr;
    int64_t *stat_pairs = nullptr;
    int32_t *stat_nrr = nullptr;
    uint32_t *done = nullptr;  // one pass: finished-workgroup counter (zero between launches)
    bool fused = false;
    int32_t bm_words = 0;
    unsigned long long *unconverged = nullptr;
};

// Enqueues one relay layer (Sec. 3.2; Sec. 4.1-4.2) on `stream`: the one
// pass, or rescoring + trigger then the reroute of the flagged rows
// compacted per head.  `profile`: bracket the launches with the profiler's
// events when profiling is on.
rr_status relay_launch(const rr_config &c, const RelayBuffers &b, int32_t layer, const void *Qc, const void *Kc,
                       int32_t *routes, uint8_t *mask, int64_t *pairs, int32_t *n_rerouted, hipStream_t stream,
                       bool profile)
{
    auto launch = [&](int kind, auto fn) { return profile ? timed(kind, stream, fn) : fn(); };
    if (b.fused) {
        // one pass: each tile rescores its rows' ledgers on its own scores,
        // flags them, and routes the flagged rows into the ledger
        rr::RouteArgs a = route_args(c, Qc, Kc);
        a.unconverged = b.unconverged;
        a.layer = layer;
        a.mode = rr::MODE_RELAY;
        a.led_routes = b.routes;
        a.led_sent = b.sent;
        a.led_build = b.build;
        a.led_age = b.age;
        a.flags = b.flags;
        a.mask_out = mask;
        a.alpha_out = b.alpha;
        a.beta_out = b.beta;
        a.gamma = c.gamma;
        a.bm_words = b.bm_words;
        a.blk_pairs = b.blk_pairs;
        a.blk_count = b.blk_count;
        a.done = b.done;
        a.stat_pairs = b.stat_pairs;
        a.stat_nrr = b.stat_nrr;
        a.pairs_out = pairs;
        a.nrr_out = n_rerouted;
        const int grid = c.n_heads * a.tiles_per_head;
        hipError_t e = launch(RR_KERNEL_RELAY, [&] { return rr::launch_route(a, c.dtype, grid, stream); });
        if (e != hipSuccess) return hip_fail(e, "relay launch");
    } else {
        rr::RescoreArgs s;
        std::memset(&s, 0, sizeof(s));
        s.Q = Qc;
        s.K = Kc;
        s.n_heads = c.n_heads;
        s.n_kv_heads = c.n_kv_heads;
        s.n_q = c.n_q;
        s.n_k = c.n_k;
        s.d = c.d;
        s.k = c.k;
        s.m = c.m;
        s.r = c.r;
        s.n_mand = c.n_sink + c.n_recent;
        s.min_reuse = c.min_reuse;
        s.gamma_rows = c.gamma_rows;
        s.causal = c.causal;
        s.layer = layer;
        rr::RescoreGeometry geo;
        rr::rescore_geometry(rows_of(c), c.n_q, c.n_k, geo);
        s.blocks_per_head = geo.blocks_per_head;
        s.rows_per_wave = geo.rows_per_wave;
        s.rows_per_block = geo.rows_per_block;
        s.dense = geo.dense ? 1 : 0;
        s.bm_words = geo.bm_words;
        s.gamma = c.gamma;
        s.led_routes = b.routes;
        s.led_sent = b.sent;
        s.led_build = b.build;
        s.led_age = b.age;
        s.flags = b.flags;
        s.mask_out = mask;
        s.alpha = b.alpha;
        s.beta = b.beta;
        s.blk_pairs = b.blk_pairs;
        s.blk_count = b.blk_count;
        s.seed_bound = b.seed_bound;
        s.seed_rmax = b.seed_rmax;
        hipError_t e = launch(RR_KERNEL_RESCORE, [&] { return rr::launch_rescore(s, c.dtype, stream); });
        if (e != hipSuccess) return hip_fail(e, "rescore launch");

        rr::RouteArgs a = route_args(c, Qc, Kc);
        a.unconverged = b.unconverged;
        a.layer = layer;
        a.mode = rr::MODE_REROUTE;
        a.led_routes = b.routes;
        a.led_sent = b.sent;
        a.led_build = b.build;
        a.led_age = b.age;
        a.flags = b.flags;
        a.blk_count = b.blk_count;
        a.blk_pairs = b.blk_pairs;
        a.rescore_bph = geo.blocks_per_head;
        a.stat_pairs = b.stat_pairs;
        a.stat_nrr = b.stat_nrr;
        a.pairs_out = pairs;
        a.nrr_out = n_rerouted;
        a.seed_bound = b.seed_bound;
        a.seed_rmax = b.seed_rmax;
        const int max_tiles = c.n_heads * a.tiles_per_head;
        const int grid8 = (max_tiles + 7) & ~7;  // a multiple of 8: per-XCD tile ranges
        const int grid = grid8 < 1024 ? grid8 : 1024;
        e = launch(RR_KERNEL_REROUTE, [&] { return rr::launch_route(a, c.dtype, grid, stream); });
        if (e != hipSuccess) return hip_fail(e, "reroute launch");
    }
    if (routes) {
        hipError_t e = hipMemcpyAsync(routes, b.routes, sizeof(int32_t) * rows_of(c) * c.k, hipMemcpyDeviceToDevice,
                                      stream);
        if (e != hipSuccess) return hip_fail(e, "route copy");
    }
    return RR_OK;
}

}  // namespace

extern "C" {

const char *rr_status_string(rr_status s)
{
    switch (s) {
    case RR_OK: return "ok";
    case RR_ERR_INVALID: return "invalid argument";
    case RR_ERR_OOM: return "out of device memory";
    case RR_ERR_HIP: return "HIP runtime error";
    case RR_ERR_STATE: return "call order violated";
    case RR_ERR_UNSUPPORTED: return "unsupported configuration";
    }
    return "unknown status";
}

const char *rr_last_error(void) { return g_err.c_str(); }

size_t rr_ledger_index_bytes(const rr_config *c)
{
    if (!c) return 0;
    return (size_t)rows_of(*c) * (size_t)(c->k + sent_width(*c)) * sizeof(int32_t);
}

rr_status rr_ledger_create(const rr_config *cfg, rr_ledger **out)
{
    if (!out) return fail(RR_ERR_INVALID, "out is NULL");
    *out = nullptr;
    rr_status st = validate(cfg, true);
    if (st != RR_OK) return st;
    rr_ledger *L = new (std::nothrow) rr_ledger;
    if (!L) return fail(RR_ERR_OOM, "host allocation failed");
    std::memset(L, 0, sizeof(*L));
    L->cfg = *cfg;
    L->rows = rows_of(*cfg);
    L->last_layer = -1;
    if (hipGetDevice(&L->device) != hipSuccess) {
        delete L;
        return fail(RR_ERR_HIP, "hipGetDevice failed");
    }
    const int64_t rows = L->rows;
    // per-workgroup partial slots of a relay layer
    const int64_t max_blocks = relay_partial_slots(*cfg);
    if ((st = alloc(&L->routes, rows * cfg->k, "routes")) != RR_OK ||
        (st = alloc(&L->sent, rows * sent_width(*cfg), "sentinels")) != RR_OK ||
        (st = alloc(&L->build, rows, "build")) != RR_OK || (st = alloc(&L->age, rows, "age")) != RR_OK ||
        (st = alloc(&L->stat_nrr, 1, "stat_nrr")) != RR_OK ||
        (st = alloc(&L->flags, rows, "flags")) != RR_OK || (st = alloc(&L->alpha, rows, "alpha")) != RR_OK ||
        (st = alloc(&L->beta, rows, "beta")) != RR_OK ||
        (st = alloc(&L->blk_pairs, max_blocks, "rescore partials")) != RR_OK ||
        (st = alloc(&L->blk_count, max_blocks, "rescore counts")) != RR_OK ||
        (st = alloc(&L->stat_pairs, 1, "stat_pairs")) != RR_OK) {
        free_all(L);
        delete L;
        return st;
    }
    // the relay schedule (one pass or split) and the split schedule's
    // threshold seeds
    const RelayPlan plan = relay_plan(*cfg);
    L->bm_words = plan.bm_words;
    L->fused = plan.fused;
    if ((L->fused && (st = alloc(&L->done, 1, "relay counter")) != RR_OK) ||
        (plan.seeds && ((st = alloc(&L->seed_bound, rows, "seed bounds")) != RR_OK ||
                        (st = alloc(&L->seed_rmax, rows, "seed maxima")) != RR_OK))) {
        free_all(L);
        delete L;
        return st;
    }
    // One-time initialisation (outside any hot path): an empty ledger.
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = hipMemset(L->routes, 0xFF, sizeof(int32_t) * rows * cfg->k);
    if (e == hipSuccess && sent_width(*cfg) > 0) e = hipMemset(L->sent, 0xFF, sizeof(int32_t) * rows * sent_width(*cfg));
    if (e == hipSuccess) e = hipMemset(L->build, 0xFF, sizeof(int32_t) * rows);
    if (e == hipSuccess) e = hipMemset(L->age, 0, sizeof(int32_t) * rows);
    if (e == hipSuccess && L->done) e = hipMemset(L->done, 0, sizeof(uint32_t));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        free_all(L);
        delete L;
        return hip_fail(e, "ledger initialisation");
    }
    *out = L;
    return RR_OK;
}

rr_status rr_ledger_destroy(rr_ledger *L)
{
    if (!L) return RR_OK;
    DeviceGuard g(L->device);
    (void)hipDeviceSynchronize();
    free_all(L);
    delete L;
    return RR_OK;
}

rr_status rr_anchor_route(rr_ledger *L, int32_t layer, const void *Qc, const void *Kc, int32_t *routes,
                          int64_t *pairs, void *hip_stream)
{
    if (!L) return fail(RR_ERR_INVALID, "ledger is NULL");
    if (!Qc || !Kc) return fail(RR_ERR_INVALID, "Qc and Kc must be device pointers");
    if (layer < 0) return fail(RR_ERR_INVALID, "layer must be >= 0");
    DeviceGuard g(L->device);
    DeviceState *ds = nullptr;
    rr_status st = device_state(&ds);
    if (st != RR_OK) return st;
    const rr_config &c = L->cfg;
    rr::RouteArgs a = route_args(c, Qc, Kc);
    a.unconverged = ds->unconverged;
    a.layer = layer;
    a.mode = rr::MODE_ANCHOR;
    a.routes_out = routes;
    a.led_routes = L->routes;
    a.led_sent = L->sent;
    a.led_build = L->build;
    a.led_age = L->age;
    a.pairs_out = pairs;
    a.pairs_value = full_pairs(c);
    const int grid = c.n_heads * a.tiles_per_head;
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = timed(RR_KERNEL_ANCHOR, stream, [&] { return rr::launch_route(a, c.dtype, grid, stream); });
    if (e != hipSuccess) return hip_fail(e, "anchor route launch");
    L->has_state = true;
    L->last_layer = layer;
    return RR_OK;
}

rr_status rr_relay_layer(rr_ledger *L, int32_t layer, const void *Qc, const void *Kc, int32_t *routes,
                         uint8_t *mask, int64_t *pairs, int32_t *n_rerouted, void *hip_stream)
{
    if (!L) return fail(RR_ERR_INVALID, "ledger is NULL");
    if (!Qc || !Kc) return fail(RR_ERR_INVALID, "Qc and Kc must be device pointers");
    if (!L->has_state) return fail(RR_ERR_STATE, "relay before any anchor or import");
    if (layer < L->last_layer) return fail(RR_ERR_STATE, "layer is below the previous call's layer");
    DeviceGuard g(L->device);
    DeviceState *ds = nullptr;
    rr_status st = device_state(&ds);
    if (st != RR_OK) return st;
    RelayBuffers b;
    b.routes = L->routes;
    b.sent = L->sent;
    b.build = L->build;
    b.age = L->age;
    b.flags = L->flags;
    b.alpha = L->alpha;
    b.beta = L->beta;
    b.seed_bound = L->seed_bound;
    b.seed_rmax = L->seed_rmax;
    b.blk_pairs = L->blk_pairs;
    b.blk_count = L->blk_count;
    b.stat_pairs = L->stat_pairs;
    b.stat_nrr = L->stat_nrr;
    b.done = L->done;
    b.fused = L->fused;
    b.bm_words = L->bm_words;
    b.unconverged = ds->unconverged;
    st = relay_launch(L->cfg, b, layer, Qc, Kc, routes, mask, pairs, n_rerouted,
                      reinterpret_cast<hipStream_t>(hip_stream), true);
    if (st != RR_OK) return st;
    L->last_layer = layer;
    return RR_OK;
}

rr_status rr_relay_layer_static(const rr_config *cfg, int32_t layer, const void *Qc, const void *Kc,
                                int32_t *led_routes, int32_t *led_sent, int32_t *led_build, int32_t *led_age,
                                int32_t *routes, uint8_t *mask, int64_t *pairs, int32_t *n_rerouted,
                                void *hip_stream)
{
    rr_status st = validate(cfg, true);
    if (st != RR_OK) return st;
    const rr_config &c = *cfg;
    if (!Qc || !Kc || !led_routes || !led_build || !led_age || (!led_sent && sent_width(c) > 0))
        return fail(RR_ERR_INVALID, "Qc, Kc and the ledger arrays (routes, sent, build, age) are required");
    if (layer < 0) return fail(RR_ERR_INVALID, "layer must be >= 0");
    RelayPlan plan = relay_plan(c);
    const StaticLayout lay = static_layout(c, plan);
    if (lay.bytes > kScratchBytes)
        return fail(RR_ERR_UNSUPPORTED, "rr_relay_layer_static: the relay scratch of this configuration (" +
                                            std::to_string(lay.bytes) + " bytes) exceeds the library's " +
                                            std::to_string(kScratchBytes) + "-byte static area");
    DeviceState *ds = nullptr;
    if ((st = device_state(&ds)) != RR_OK) return st;
    unsigned char *base = ds->scratch;
    RelayBuffers b;
    b.routes = led_routes;
    b.sent = led_sent;
    b.build = led_build;
    b.age = led_age;
    b.done = reinterpret_cast<uint32_t *>(base + lay.done);
    b.stat_pairs = reinterpret_cast<int64_t *>(base + lay.stat_pairs);
    b.stat_nrr = reinterpret_cast<int32_t *>(base + lay.stat_nrr);
    b.blk_pairs = reinterpret_cast<int64_t *>(base + lay.blk_pairs);
    b.blk_count = reinterpret_cast<int32_t *>(base + lay.blk_count);
    b.flags = base + lay.flags;
    b.alpha = reinterpret_cast<float *>(base + lay.alpha);
    b.beta = reinterpret_cast<float *>(base + lay.beta);
    b.seed_bound = plan.seeds ? reinterpret_cast<float *>(base + lay.seed_bound) : nullptr;
    b.seed_rmax = plan.seeds ? reinterpret_cast<float *>(base + lay.seed_rmax) : nullptr;
    b.fused = plan.fused;
    b.bm_words = plan.bm_words;
    b.unconverged = ds->unconverged;
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    if (plan.fused) {
        // the one pass's completion counter must read zero at launch: the
        // area keeps the previous call's contents, so it is cleared here, on
        // the caller's stream, by a kernel (a stream under capture records a
        // plain kernel node, not a memset)
        hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(64), 0, stream, b.done, 1);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "relay scratch clear");
    }
    return relay_launch(c, b, layer, Qc, Kc, routes, mask, pairs, n_rerouted, stream, false);
}

rr_status rr_full_route(const rr_config *cfg, const void *Qc, const void *Kc, int32_t *routes, float *route_scores,
                        int64_t *pairs, void *hip_stream)
{
    rr_status st = validate(cfg, false);
    if (st != RR_OK) return st;
    if (!Qc || !Kc || !routes) return fail(RR_ERR_INVALID, "Qc, Kc and routes must be device pointers");
    DeviceState *ds = nullptr;
    if ((st = device_state(&ds)) != RR_OK) return st;
    rr_config c = *cfg;
    c.m = 0;
    c.r = 0;
    c.n_sink = 0;
    c.n_recent = 0;
    rr::RouteArgs a = route_args(c, Qc, Kc);
    a.unconverged = ds->unconverged;
    a.mode = rr::MODE_FULL;
    a.routes_out = routes;
    a.scores_out = route_scores;
    a.pairs_out = pairs;
    a.pairs_value = full_pairs(c);
    const int grid = c.n_heads * a.tiles_per_head;
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = timed(RR_KERNEL_FULL, stream, [&] { return rr::launch_route(a, c.dtype, grid, stream); });
    if (e != hipSuccess) return hip_fail(e, "full route launch");
    return RR_OK;
}

const int32_t *rr_ledger_routes(const rr_ledger *L) { return L ? L->routes : nullptr; }

rr_status rr_ledger_export(const rr_ledger *L, int32_t *routes, int32_t *sent, int32_t *build, int32_t *age,
                           void *hip_stream)
{
    if (!L) return fail(RR_ERR_INVALID, "ledger is NULL");
    DeviceGuard g(L->device);
    hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    const rr_config &c = L->cfg;
    hipError_t e = hipSuccess;
    if (routes) e = hipMemcpyAsync(routes, L->routes, sizeof(int32_t) * L->rows * c.k, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && sent && sent_width(c) > 0)
        e = hipMemcpyAsync(sent, L->sent, sizeof(int32_t) * L->rows * sent_width(c), hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && build) e = hipMemcpyAsync(build, L->build, sizeof(int32_t) * L->rows, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && age) e = hipMemcpyAsync(age, L->age, sizeof(int32_t) * L->rows, hipMemcpyDeviceToDevice, s);
    return e == hipSuccess ? RR_OK : hip_fail(e, "ledger export");
}

rr_status rr_ledger_import(rr_ledger *L, int32_t layer, const int32_t *routes, const int32_t *sent,
                           const int32_t *build, const int32_t *age, void *hip_stream)
{
    if (!L) return fail(RR_ERR_INVALID, "ledger is NULL");
    const rr_config &c = L->cfg;
    if (!routes || !build || !age || (!sent && sent_width(c) > 0))
        return fail(RR_ERR_INVALID, "routes, sent, build and age are required");
    if (layer < 0) return fail(RR_ERR_INVALID, "layer must be >= 0");
    DeviceGuard g(L->device);
    hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = hipMemcpyAsync(L->routes, routes, sizeof(int32_t) * L->rows * c.k, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && sent_width(c) > 0)
        e = hipMemcpyAsync(L->sent, sent, sizeof(int32_t) * L->rows * sent_width(c), hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(L->build, build, sizeof(int32_t) * L->rows, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(L->age, age, sizeof(int32_t) * L->rows, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "ledger import");
    L->has_state = true;
    L->last_layer = layer;
    return RR_OK;
}

rr_status rr_ledger_relay_stats(const rr_ledger *L, float *alpha, float *beta, int32_t *ids, void *hip_stream)
{
    if (!L) return fail(RR_ERR_INVALID, "ledger is NULL");
    DeviceGuard g(L->device);
    hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = hipSuccess;
    if (alpha) e = hipMemcpyAsync(alpha, L->alpha, sizeof(float) * L->rows, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && beta) e = hipMemcpyAsync(beta, L->beta, sizeof(float) * L->rows, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && ids) {
        hipLaunchKernelGGL(flagged_ids_kernel, dim3(L->cfg.n_heads), dim3(kIdsThreads), 0, s, L->flags, L->cfg.n_q, ids);
        e = hipGetLastError();
    }
    return e == hipSuccess ? RR_OK : hip_fail(e, "relay stats");
}

rr_status rr_profile_start(void)
{
    for (ProfRecord &r : g_prof.records) {
        g_prof.pool.push_back(r.start);
        g_prof.pool.push_back(r.stop);
    }
    g_prof.records.clear();
    g_prof.on = true;
    return RR_OK;
}

rr_status rr_profile_stop(double *total_ms, int64_t *launches, int32_t n_kinds)
{
    if ((total_ms || launches) && n_kinds < RR_KERNEL_KINDS)
        return fail(RR_ERR_INVALID, "rr_profile_stop: the arrays must hold RR_KERNEL_KINDS entries");
    g_prof.on = false;
    double ms[RR_KERNEL_KINDS] = {};
    int64_t n[RR_KERNEL_KINDS] = {};
    rr_status st = RR_OK;
    for (ProfRecord &r : g_prof.records) {
        hipError_t e = hipEventSynchronize(r.stop);
        float t = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, r.start, r.stop);
        if (e != hipSuccess) {
            st = hip_fail(e, "profile event");
            continue;
        }
        ms[r.kind] += t;
        n[r.kind] += 1;
    }
    for (int k = 0; k < RR_KERNEL_KINDS; ++k) {
        if (total_ms) total_ms[k] = ms[k];
        if (launches) launches[k] = n[k];
    }
    return st;
}

rr_status rr_unconverged_rows(uint64_t *count)
{
    if (!count) return fail(RR_ERR_INVALID, "count is NULL");
    DeviceState *ds = nullptr;
    rr_status st = device_state(&ds);
    if (st != RR_OK) return st;
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(count, ds->unconverged, sizeof(uint64_t), hipMemcpyDeviceToHost);
    return e == hipSuccess ? RR_OK : hip_fail(e, "unconverged-row count");
}

rr_status rr_set_sweep_cap(int32_t cap)
{
    if (cap < 0) return fail(RR_ERR_INVALID, "the sweep cap must be >= 0 (0: the default)");
    g_sweep_cap.store(cap, std::memory_order_relaxed);
    return RR_OK;
}

}  // extern "C"

// ------------------------------------------------- either side of the path

rr_status rr_pool_chunks(const void *X, int32_t n_heads, int32_t n_tokens, int32_t d, int32_t chunk,
                         int32_t dtype, void *Xc, void *hip_stream)
{
    if (!X || !Xc) return fail(RR_ERR_INVALID, "X and Xc must be device pointers");
    if (n_heads < 1 || n_tokens < 1 || chunk < 1) return fail(RR_ERR_INVALID, "n_heads, n_tokens and chunk must be >= 1");
    if (d < 8 || d > 1024 || d % 8 != 0) return fail(RR_ERR_INVALID, "d must be a multiple of 8 in [8, 1024]");
    if (dtype != RR_F32 && dtype != RR_BF16) return fail(RR_ERR_INVALID, "unknown dtype");
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = timed(RR_KERNEL_POOL, stream,
                         [&] { return rr::launch_pool(X, n_heads, n_tokens, d, chunk, dtype, Xc, stream); });
    return e == hipSuccess ? RR_OK : hip_fail(e, "pooling launch");
}

rr_status rr_expand_tokens(const int32_t *routes, int64_t rows, int32_t k, int32_t chunk, int32_t n_tokens,
                           int32_t *tokens, void *hip_stream)
{
    if (!routes || !tokens) return fail(RR_ERR_INVALID, "routes and tokens must be device pointers");
    if (rows < 1 || k < 1 || chunk < 1 || n_tokens < 1)
        return fail(RR_ERR_INVALID, "rows, k, chunk and n_tokens must be >= 1");
    if ((int64_t)k * chunk > INT32_MAX) return fail(RR_ERR_INVALID, "k * chunk beyond int32");
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = timed(RR_KERNEL_EXPAND, stream,
                         [&] { return rr::launch_expand(routes, rows, k, chunk, n_tokens, tokens, stream); });
    return e == hipSuccess ? RR_OK : hip_fail(e, "expansion launch");
}

rr_status rr_sparse_attention(const rr_attn_config *cfg, const void *Q, const void *K, const void *V,
                              const int32_t *routes, void *O, void *hip_stream)
{
    if (!cfg) return fail(RR_ERR_INVALID, "config is NULL");
    const rr_attn_config &c = *cfg;
    if (!Q || !K || !V || !routes || !O) return fail(RR_ERR_INVALID, "Q, K, V, routes and O must be device pointers");
    if (c.n_heads < 1 || c.n_kv_heads < 1 || c.n_heads % c.n_kv_heads != 0)
        return fail(RR_ERR_INVALID, "n_heads must be a positive multiple of n_kv_heads");
    if (c.n_tokens < 1 || c.chunk < 1) return fail(RR_ERR_INVALID, "n_tokens and chunk must be >= 1");
    if (c.k < 1 || c.k > rr::kMaxAttnSlots) return fail(RR_ERR_INVALID, "k must lie in [1, 256]");
    if (c.causal != 0 && c.causal != 1) return fail(RR_ERR_INVALID, "causal must be 0 or 1");
    if (c.reserved != 0) return fail(RR_ERR_INVALID, "rr_attn_config.reserved must be 0");
    if (!(c.scale >= 0.f) || std::isinf(c.scale)) return fail(RR_ERR_INVALID, "scale must be finite and >= 0");
    if (c.dtype != RR_F32 && c.dtype != RR_BF16) return fail(RR_ERR_INVALID, "unknown dtype");
    if (!rr::attention_supported(c.dtype, c.d))
        return fail(RR_ERR_UNSUPPORTED, "sparse attention supports bf16 with d = 64 or 128");
    rr::AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.Q = Q;
    a.K = K;
    a.V = V;
    a.O = O;
    a.routes = routes;
    a.n_heads = c.n_heads;
    a.n_kv_heads = c.n_kv_heads;
    a.n_tokens = c.n_tokens;
    a.d = c.d;
    a.chunk = c.chunk;
    a.k = c.k;
    a.causal = c.causal;
    a.n_chunks = (int32_t)(((int64_t)c.n_tokens + c.chunk - 1) / c.chunk);
    a.tiles_per_chunk = rr::attention_tiles_per_chunk(c.chunk < c.n_tokens ? c.chunk : c.n_tokens);
    a.scale = c.scale > 0.f ? c.scale : 1.f / std::sqrt((float)c.d);
    if ((int64_t)c.n_heads * a.n_chunks * a.tiles_per_chunk > INT32_MAX)
        return fail(RR_ERR_INVALID, "too many query tiles");
    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = timed(RR_KERNEL_ATTENTION, stream, [&] { return rr::launch_attention(a, stream); });
    return e == hipSuccess ? RR_OK : hip_fail(e, "attention launch");
}
