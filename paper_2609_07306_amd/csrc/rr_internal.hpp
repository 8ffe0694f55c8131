// Route kernel argument block and launchers shared by the host API and the
// kernels (the rescoring kernels' are in rr_rescore.hpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace rr {

enum RouteMode : int32_t {
    MODE_FULL = 0,     // stateless routing, k slots, no sentinels
    MODE_ANCHOR = 1,   // every row: route + near-miss + random sentinels -> ledger
    MODE_REROUTE = 2,  // flagged rows only (compacted per head) -> ledger
    MODE_RELAY = 3,    // every row rescored against the ledger on the tile's own
                       // scores, then the flagged rows routed -> ledger
};

constexpr int kNarrowTileRows = 128;  // route tile rows when k + m <= 64
constexpr int kWideTileRows = 64;     // route tile rows when 64 < k + m <= 128
constexpr int kSmallTileRows = 32;    // route tile rows when k + m <= 64 and 128-row tiles would be few
constexpr int kFewTiles = 256;        // ... fewer than this many (one per compute unit)

struct RouteArgs {
    const void *Q;
    const void *K;
    int32_t n_heads, n_kv_heads, n_q, n_k, d;
    int32_t k, m, r;  // the kernel selects T = k + m chunks per row
    int32_t n_sink, n_recent;  // mandatory sentinels (sentinel slots: m near-miss, r random, n_sink + n_recent mandatory)
    int32_t min_reuse;         // relay: minimum reuse horizon in layers (0: none)
    const float *gamma_rows;   // relay: per-row guard margins, or null (gamma for every row)
    const int32_t *k_rows;     // per-row route widths in [1, k] (clamped), or null (k for every row)
    int32_t causal;
    int32_t layer;
    int32_t mode;
    int32_t tile_rows;       // route_tile_rows() of the call's shape
    int32_t tiles_per_head;  // ceil(n_q / tile rows) for full / anchor tiles
    int32_t lds_region0;     // set by the launcher: bytes of the key-tile region
    uint64_t seed;
    int32_t *routes_out;  // [rows, k] or null
    float *scores_out;    // [rows, k] or null
    int32_t *led_routes;  // ledger (anchor / reroute)
    int32_t *led_sent;
    int32_t *led_build;
    int32_t *led_age;
    uint8_t *flags;            // reroute: [rows] (relay: written)
    int32_t *blk_count;        // reroute: flagged rows per rescoring workgroup, head-major (relay: per tile)
    int64_t *blk_pairs;        // reroute: score pairs per rescoring workgroup, head-major (relay: per tile)
    int32_t rescore_bph;       // reroute: rescoring workgroups per head
    int32_t lds_tiles;         // reroute: LDS byte offset of the per-head tile table (set by the launcher)
    int64_t *stat_pairs;       // reroute: the call's score pairs (ledger copy)
    int32_t *stat_nrr;         // reroute: the call's rerouted rows (ledger copy)
    int32_t *nrr_out;          // reroute: optional device scalar
    const float *seed_bound;   // reroute, or null: per row, a lower bound of its T-th score ...
    const float *seed_rmax;    // ... and its largest score, from the rescoring pass (no threshold sweep)
    uint8_t *mask_out;         // relay: [rows] caller mask or null
    float *alpha_out;          // relay: [rows] min over R of the rescored scores
    float *beta_out;           // relay: [rows] max over C
    float gamma;               // relay: guard margin
    int32_t bm_words;          // relay: ledger bitmap row stride in (R, C) word pairs
    uint32_t *done;            // relay: finished-workgroup counter (0 between launches)
    int64_t *pairs_out;        // optional device scalar
    int64_t pairs_value;       // value written to pairs_out (full / anchor; reroute: the workgroup sums)
    unsigned long long *unconverged;  // device counter: rows whose collection stopped at the sweep cap
    int32_t sweep_cap;                // collection sweeps allowed per tile (kMaxFixIters unless a test lowers it)
};

// Raises a kernel's dynamic LDS limit on the current device when a launch
// needs more than any earlier one there (the default limit is 64 KiB), so
// the runtime call is made once per kernel instance and device rather than
// on every launch.  `seen` is the instance's own record, zero-initialised.
struct LdsLimit {
    std::atomic<int> bytes[64];
};

inline hipError_t raise_lds_limit(const void *fn, size_t lds, LdsLimit &seen)
{
    if (lds <= 65536) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64 && seen.bytes[dev].load(std::memory_order_acquire) >= (int)lds) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess && dev >= 0 && dev < 64) {
        int cur = seen.bytes[dev].load(std::memory_order_relaxed);
        while (cur < (int)lds && !seen.bytes[dev].compare_exchange_weak(cur, (int)lds)) {
        }
    }
    return e;
}


// Sparse attention over routed chunks (rr_consumer.hip).
constexpr int kMaxAttnSlots = 256;  // route slots per row

struct AttnArgs {
    const void *Q, *K, *V;  // bf16 [H, n_tokens, d], [H_kv, n_tokens, d] x2
    void *O;                // bf16 [H, n_tokens, d]
    const int32_t *routes;  // [H * n_chunks, k]
    int32_t n_heads, n_kv_heads, n_tokens, d, chunk, k, causal;
    int32_t n_chunks, tiles_per_chunk;
    float scale;
};

bool attention_supported(int dtype, int d);
int attention_tiles_per_chunk(int chunk);
hipError_t launch_attention(const AttnArgs &a, hipStream_t stream);
hipError_t launch_pool(const void *X, int n_heads, int n_tok, int d, int chunk, int dtype, void *out,
                       hipStream_t stream);
hipError_t launch_expand(const int32_t *routes, int64_t rows, int k, int chunk, int n_tok, int32_t *tokens,
                         hipStream_t stream);

// Supported (dtype, d) combinations; dtype 0 = binary32, 1 = bf16.
bool route_supported(int dtype, int d, int T);
int route_tile_rows(int T, int n_heads, int n_q);  // query rows per route tile for T = k + m
// Largest ledger bitmap (word pairs per row) a relay tile holds in LDS.
int route_relay_max_bm_words(int dtype, int d, int T);
hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream);

}  // namespace rr
