// Kernel argument blocks and launchers shared by the host API and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rr {

enum RouteMode : int32_t {
    MODE_FULL = 0,     // stateless routing, k slots, no sentinels
    MODE_ANCHOR = 1,   // every row: route + near-miss + random sentinels -> ledger
    MODE_REROUTE = 2,  // flagged rows only (compacted per head) -> ledger
};

constexpr int kNarrowTileRows = 128;  // route tile rows when k + m <= 64
constexpr int kWideTileRows = 64;     // route tile rows when 64 < k + m <= 128
constexpr int kRescoreWaves = 4;            // waves per rescoring workgroup
constexpr int kRescoreBlocks = 512;         // target rescoring workgroups per launch (two per CU)
constexpr int kRescoreMaxRowsPerWave = 16;  // rows a rescoring wave scores in turn
constexpr int kRescoreLanesPerCand = 4;     // lanes sharing one candidate's dot product (4 or 8)
constexpr int kRescoreDenseMaxKeys = 2048;  // dense (MFMA tile) rescoring up to this many key chunks
constexpr int kRescoreDenseMinTiles = 256;  // ... and with at least this many 128-row tiles (one per CU)

struct RouteArgs {
    const void *Q;
    const void *K;
    int32_t n_heads, n_kv_heads, n_q, n_k, d;
    int32_t k, m, r;  // the kernel selects T = k + m chunks per row
    int32_t causal;
    int32_t layer;
    int32_t mode;
    int32_t tiles_per_head;  // ceil(n_q / tile rows) for full / anchor tiles
    int32_t lds_region0;     // set by the launcher: bytes of the key-tile region
    uint64_t seed;
    int32_t *routes_out;  // [rows, k] or null
    float *scores_out;    // [rows, k] or null
    int32_t *led_routes;  // ledger (anchor / reroute)
    int32_t *led_sent;
    int32_t *led_build;
    int32_t *led_age;
    const uint8_t *flags;      // reroute: [rows]
    const int32_t *blk_count;  // reroute: flagged rows per rescoring workgroup, head-major
    const int64_t *blk_pairs;  // reroute: score pairs per rescoring workgroup, head-major
    int32_t rescore_bph;       // reroute: rescoring workgroups per head
    int32_t lds_tiles;         // reroute: LDS byte offset of the per-head tile table (set by the launcher)
    int64_t *stat_pairs;       // reroute: the call's score pairs (ledger copy)
    int32_t *stat_nrr;         // reroute: the call's rerouted rows (ledger copy)
    int32_t *nrr_out;          // reroute: optional device scalar
    int32_t *ids_out;          // reroute: compacted row ids per head, or null
    int64_t *pairs_out;        // optional device scalar
    int64_t pairs_value;       // value written to pairs_out (full / anchor; reroute: the workgroup sums)
};

struct RescoreArgs {
    const void *Q;
    const void *K;
    int32_t n_heads, n_kv_heads, n_q, n_k, d;
    int32_t k, m, r;
    int32_t causal;
    int32_t layer;
    int32_t blocks_per_head;  // ceil(n_q / rows per block)
    int32_t rows_per_wave;    // gather: rows per block = kRescoreWaves * rows_per_wave
    int32_t dense;            // 1: the MFMA tile kernel (128-row tiles), 0: the gather kernel
    int32_t bm_words;         // dense: bitmap row stride in (R, C) word pairs (padded key range + 1, odd)
    float gamma;
    const int32_t *led_routes;
    const int32_t *led_sent;
    const int32_t *led_build;
    int32_t *led_age;
    uint8_t *flags;     // [rows] internal reroute flags
    uint8_t *mask_out;  // [rows] caller mask or null
    float *alpha;
    float *beta;
    int64_t *blk_pairs;  // [n_heads * blocks_per_head] score pairs per workgroup (head-major)
    int32_t *blk_count;  // [n_heads * blocks_per_head] flagged rows per workgroup
};

// Supported (dtype, d) combinations; dtype 0 = binary32, 1 = bf16.
bool route_supported(int dtype, int d, int T);
int route_tile_rows(int T);  // query rows per route tile for T = k + m
hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream);
// Launch shape of the rescoring kernel for a configuration.
struct RescoreGeometry {
    int rows_per_wave, rows_per_block, blocks_per_head;
    bool dense;
    int bm_words;
};
void rescore_geometry(int64_t rows, int n_q, int n_k, RescoreGeometry &g);
hipError_t launch_rescore(const RescoreArgs &a, int dtype, hipStream_t stream);
int rescore_dense_tile_rows();
hipError_t launch_rescore_dense(const RescoreArgs &a, int dtype, hipStream_t stream);

}  // namespace rr
