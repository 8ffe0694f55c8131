// Rescoring kernel argument block, tuning constants and launchers shared by
// the host API and the two rescoring kernels (dense MFMA tiles, L2 gather).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rr {

constexpr int kRescoreWaves = 4;            // waves per rescoring workgroup
constexpr int kRescoreBlocks = 512;         // target rescoring workgroups per launch (two per CU)
constexpr int kRescoreMaxRowsPerWave = 16;  // rows a rescoring wave scores in turn
constexpr int kRescoreLanesPerCand = 4;     // lanes sharing one candidate's dot product (4 or 8)
constexpr int kRescoreDenseMaxKeys = 2048;  // dense (MFMA tile) rescoring up to this many key chunks
constexpr int kDenseRowsLarge = 128;        // dense tile rows with at least kRescoreDenseFullTiles such tiles
constexpr int kDenseRowsSmall = 64;         // ... else, with at least kRescoreDenseMinTiles of these
constexpr int kRescoreDenseFullTiles = 256;  // a tile per compute unit
constexpr int kRescoreDenseMinTiles = 128;   // half the compute units

struct RescoreArgs {
    const void *Q;
    const void *K;
    int32_t n_heads, n_kv_heads, n_q, n_k, d;
    int32_t k, m, r;
    int32_t n_mand;           // mandatory sentinel slots after the random ones
    int32_t min_reuse;        // minimum reuse horizon in layers (0: none)
    const float *gamma_rows;  // per-row guard margins, or null (gamma for every row)
    int32_t causal;
    int32_t layer;
    int32_t blocks_per_head;  // ceil(n_q / rows per block)
    int32_t rows_per_wave;    // gather: rows per block = kRescoreWaves * rows_per_wave
    int32_t rows_per_block;   // dense: tile rows (kDenseRowsLarge or kDenseRowsSmall)
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
    float *seed_bound;   // dense, or null: [rows] a lower bound of the row's (k+m)-th score
    float *seed_rmax;    // dense, or null: [rows] the row's largest score
};

// Launch shape of the rescoring kernel for a configuration.
struct RescoreGeometry {
    int rows_per_wave, rows_per_block, blocks_per_head;
    bool dense;
    int bm_words;
};
void rescore_geometry(int64_t rows, int n_q, int n_k, RescoreGeometry &g);
hipError_t launch_rescore(const RescoreArgs &a, int dtype, hipStream_t stream);
bool rescore_dense_seeds(int dtype, int d);  // the dense kernel writes seed_bound / seed_rmax
hipError_t launch_rescore_dense(const RescoreArgs &a, int dtype, hipStream_t stream);

}  // namespace rr
