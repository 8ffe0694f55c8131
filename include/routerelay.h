/*
 * routerelay.h -- C ABI of librouterelay.so, the MI355X (gfx950) route-
 * maintenance path of RouteRelay (arXiv 2609.07306).
 *
 * Problem (Sec. 2.1, Eq. (1)-(2)): per query head h, chunk representations
 * Qc[h] in R^{n_q x d} and Kc[g] in R^{n_k x d} (g = h / (H_q / H_kv)) give
 * scores S = Qc Kc^T, and row i routes to the k best key chunks.  RouteRelay
 * (Sec. 3) keeps, per row, a ledger of the selected set R, m near-miss and r
 * random sentinels C, and the layer the entry was built at.  Anchor layers
 * rebuild every entry; intermediate (relay) layers rescore R u C, keep the
 * route of a row when its weakest selected score beats its strongest sentinel
 * by more than gamma, and fully reroute the other rows only (Sec. 3.2,
 * Sec. 4.1-4.2).
 *
 * Conventions shared by every call:
 *   - Tensors are DEVICE pointers owned by the caller, row-major, contiguous.
 *     Qc is [H_q, n_q, d] and Kc is [H_kv, n_k, d], binary32 (RR_F32) or bf16
 *     (RR_BF16, 16-bit storage).  Scores are accumulated in binary32.
 *   - Row index: row = h * n_q + i.  The causal chunk mask lets row i select
 *     key chunks j <= i only (needs n_q == n_k); such a row has n_i = i + 1
 *     valid chunks, a row without the mask has n_i = n_k.
 *   - A route is a SET, stored sorted by ascending chunk id and padded with
 *     -1 (a row with n_i < k routes to all of its valid chunks).  Ties in
 *     score are broken toward the lower chunk id; -0 equals +0.
 *   - Every call enqueues work on the given HIP stream (NULL: the null
 *     stream) and returns; outputs, including device counters, are valid once
 *     that stream has reached the enqueued work.  No call synchronises the
 *     host with the device and none allocates memory, except
 *     rr_ledger_create.
 *   - The caller keeps Qc, Kc and the output buffers alive until the stream
 *     has passed the call.  A ledger is used by one host thread on one stream
 *     at a time.
 *   - Errors are reported by the return value; rr_last_error() returns a
 *     message for the calling thread's most recent failure.  Argument errors
 *     are detected before any work is enqueued.
 */
#ifndef ROUTERELAY_H
#define ROUTERELAY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RR_OK = 0,
    RR_ERR_INVALID = -1,     /* an argument or configuration value is invalid */
    RR_ERR_OOM = -2,         /* device allocation failed */
    RR_ERR_HIP = -3,         /* a HIP runtime call failed (message in rr_last_error) */
    RR_ERR_STATE = -4,       /* call order violated (relay before any anchor, layer going back) */
    RR_ERR_UNSUPPORTED = -5  /* valid but outside the shapes the library supports */
} rr_status;

typedef enum { RR_F32 = 0, RR_BF16 = 1 } rr_dtype;

/* Shape and rule parameters.  Supported: d in {32, 64, 128} (and 256 for
 * bf16); 1 <= k <= n_k; k + m <= 128; k + m + r + n_sink + n_recent <= 256;
 * n_k <= 8192;
 * n_heads a multiple of n_kv_heads; gamma not NaN.  gamma is the guard
 * margin of Eq. (8); the paper uses gamma >= 0 (0 by default, Table 1);
 * +INFINITY refreshes every row that has a sentinel and -INFINITY refreshes
 * none.  seed keys the random-sentinel probes. */
/* Options (rr_config.options).  A relay layer (Sec. 3.2) runs as one of two
 * schedules with the same results:
 *   one pass -- over the 128-row (or 64-row) tiles of every head, the tile's
 *     scores rescore its rows' ledgers, the trigger flags rows, and the same
 *     pass routes the flagged ones (possible while a tile's ledger bitmaps
 *     fit its LDS: n_k up to about 2048, d = 256 up to about 1900);
 *   split -- rescoring and trigger, then the routing of the flagged rows
 *     compacted per head (Sec. 4.2).
 * By default causal inputs take the one pass where it fits (compaction would
 * mix short and long causal rows in one tile) and other inputs the split
 * schedule, measured faster for them.  RR_OPT_SPLIT_RELAY forces the split
 * schedule, RR_OPT_ONE_PASS_RELAY the one pass (RR_ERR_UNSUPPORTED where it
 * does not fit); not both. */
typedef enum { RR_OPT_SPLIT_RELAY = 1, RR_OPT_ONE_PASS_RELAY = 2 } rr_option;

typedef struct {
    int32_t n_heads;    /* H_q */
    int32_t n_kv_heads; /* H_kv */
    int32_t n_q;        /* query chunks per head */
    int32_t n_k;        /* key chunks per head */
    int32_t d;          /* representation width */
    int32_t k;          /* route width */
    int32_t m;          /* near-miss sentinels */
    int32_t r;          /* random sentinels */
    int32_t dtype;      /* rr_dtype of Qc and Kc */
    int32_t causal;     /* 1: chunk mask j <= i */
    float gamma;        /* guard margin */
    uint32_t options;   /* rr_option bits (0: defaults) */
    uint64_t seed;
    /* Mandatory sentinels (Sec. 3.1, item 3): the sink chunks j < n_sink and
     * the recent chunks -- the n_recent valid chunks up to the row's position
     * (row i when n_q == n_k, else the last key chunk) -- that are not in R or
     * N, kept ascending in n_sink + n_recent extra sentinel slots after the
     * random ones (-1 padded) and left out of the random draws. */
    int32_t n_sink;
    int32_t n_recent;
    /* Minimum reuse horizon (Sec. 3.2, Hysteresis): a row (re)built at layer
     * b is not rerouted at layers b+1 .. b+min_reuse.  0: off. */
    int32_t min_reuse;
    int32_t reserved;           /* must be 0 */
    /* Per-row guard margins gamma_i of Eq. (8): a device array of H_q*n_q
     * binary32 values read by every relay (the caller may change them between
     * layers, e.g. to raise the margin of recently refreshed rows); NULL: the
     * scalar gamma for every row.  Values must not be NaN. */
    const float *gamma_rows;
    /* Query-dependent route budgets (Sec. 4.3): a device array of H_q*n_q
     * int32 route widths k_i, read by every routing call (full, anchor,
     * relay).  Row i routes to its k_i best chunks, in its first k_i route
     * slots (the other k - k_i are -1), and its near-miss sentinels are the m
     * chunks ranked after them.  Rows of every width share the launches (one
     * bucket).  Values outside [1, k] are clamped to it.  NULL: k for every
     * row. */
    const int32_t *k_rows;
} rr_config;

typedef struct rr_ledger rr_ledger;

/* Route ledger (Sec. 3.1, Eq. (4); state tensors of Sec. 4.1).  Allocates,
 * on the current HIP device, the structure-of-arrays ledger -- routes
 * [H_q*n_q, k], sentinels [H_q*n_q, m+r+n_sink+n_recent] (near-miss slots
 * first, sorted by id; then random slots in draw order; then mandatory slots,
 * sorted by id; -1 padded), build layer and age
 * [H_q*n_q] int32 -- plus the per-row scratch of the relay path.  *out
 * receives the handle (NULL on failure).  Returns RR_ERR_INVALID /
 * RR_ERR_UNSUPPORTED for a bad config, RR_ERR_OOM if allocation fails. */
rr_status rr_ledger_create(const rr_config *cfg, rr_ledger **out);

/* Frees the ledger's device memory after synchronising the device.  NULL is
 * a no-op. */
rr_status rr_ledger_destroy(rr_ledger *ledger);

/* Anchor layer (Sec. 3.1; forced anchors, Sec. 3.2): full routing of every
 * row (Eq. (1)-(2)) that also keeps the chunks ranked k+1..k+m as near-miss
 * sentinels and draws r random sentinels from the remaining valid chunks;
 * every ledger entry is rebuilt with build layer = layer and age 0.
 *   layer   >= 0; it keys the random probes.  An anchor may restart the layer
 *           sequence (a new forward pass): later relays must not go below it.
 *   Qc, Kc  device inputs as above.
 *   routes  optional device output [H_q*n_q, k] int32 (a copy of the ledger's
 *           routes); may be NULL.
 *   pairs   optional device int64: number of scores evaluated (sum of n_i).
 */
rr_status rr_anchor_route(rr_ledger *ledger, int32_t layer, const void *Qc, const void *Kc,
                          int32_t *routes, int64_t *pairs, void *hip_stream);

/* Relay layer (Sec. 3.2, Eq. (5)-(8); dataflow of Sec. 4.1-4.2).  Each row
 * rescores its candidates A = R u C at this layer: alpha = min over R,
 * beta = max over C.  A row with a non-empty C and beta + gamma >= alpha is
 * rerouted: its full score row is computed and its ledger entry rebuilt as at
 * an anchor (build layer = layer, age 0).  Other rows keep their entry and get
 * age = layer - build layer.  Only the rerouted rows run the selection and
 * the ledger rebuild: compacted per head for a second launch (split
 * schedule), or within the rescoring launch's own tiles (one-pass schedule);
 * rr_config.options and the inputs choose the schedule, the results are the
 * same.
 *   routes      optional device output [H_q*n_q, k] int32 (copy of the
 *               ledger's routes after the update); NULL to read the ledger
 *               through rr_ledger_routes instead.
 *   mask        optional device output [H_q*n_q] uint8: 1 = rerouted.
 *   pairs       optional device int64: scores evaluated, i.e. the sum over
 *               rows of |A_i| (valid candidate slots) plus n_i per rerouted
 *               row.
 *   n_rerouted  optional device int32: number of rerouted rows.
 * Returns RR_ERR_STATE if no anchor (or import) preceded it or if layer is
 * below the previous call's layer. */
rr_status rr_relay_layer(rr_ledger *ledger, int32_t layer, const void *Qc, const void *Kc,
                         int32_t *routes, uint8_t *mask, int64_t *pairs, int32_t *n_rerouted,
                         void *hip_stream);

/* Relay layer that allocates nothing, for callers that cannot allocate
 * device memory at call time: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  The same computation and kernels as
 * rr_relay_layer, on a ledger the caller owns, in the layout rr_ledger_export
 * writes: led_routes [H_q*n_q, k], led_sent [H_q*n_q, m+r+n_sink+n_recent]
 * (may be NULL when that width is 0), led_build and led_age [H_q*n_q]
 * int32, all device memory,
 * updated in place.  The relay's scratch (flags, alpha / beta, per-workgroup
 * partials, call totals, threshold seeds, a completion counter) lives in a
 * static device area of the library, 4 MiB per GPU, held until the process
 * ends; a configuration whose scratch exceeds it (beyond about 200 000 routed
 * rows) returns RR_ERR_UNSUPPORTED before any work is enqueued.  There is no
 * call-order state: the caller keeps layers non-decreasing after an anchor
 * built the ledger.  Every call on one GPU shares that GPU's area, so calls
 * that overlap on one GPU (concurrent streams or threads) race; calls
 * ordered on one stream do not.  routes, mask, pairs and n_rerouted are as in
 * rr_relay_layer. */
rr_status rr_relay_layer_static(const rr_config *cfg, int32_t layer, const void *Qc, const void *Kc,
                                int32_t *led_routes, int32_t *led_sent, int32_t *led_build,
                                int32_t *led_age, int32_t *routes, uint8_t *mask, int64_t *pairs,
                                int32_t *n_rerouted, void *hip_stream);

/* Full routing baseline (Eq. (1)-(2)) with the same GEMM + TopK kernels and
 * no ledger: routes [H_q*n_q, cfg->k] int32 receives every row's route.
 * cfg->m and cfg->r are ignored.  route_scores (optional, [H_q*n_q, k]
 * binary32) receives the score of each route slot (padding: -INFINITY).
 * pairs (optional device int64) receives the number of scores evaluated. */
rr_status rr_full_route(const rr_config *cfg, const void *Qc, const void *Kc, int32_t *routes,
                        float *route_scores, int64_t *pairs, void *hip_stream);

/* Borrowed device view of the ledger's routes [H_q*n_q, k]; valid until the
 * next call that mutates or destroys the ledger.  NULL for a NULL ledger. */
const int32_t *rr_ledger_routes(const rr_ledger *ledger);

/* Copies the ledger state into caller device buffers (each may be NULL):
 * routes [rows,k], sent [rows,m+r+n_sink+n_recent], build [rows], age [rows]
 * int32. */
rr_status rr_ledger_export(const rr_ledger *ledger, int32_t *routes, int32_t *sent,
                           int32_t *build, int32_t *age, void *hip_stream);

/* Replaces the ledger state from caller device buffers (all four required)
 * and records `layer` as the last layer seen, so that a relay may follow.
 * The contents are trusted: ids must lie in [-1, n_i) with R sorted. */
rr_status rr_ledger_import(rr_ledger *ledger, int32_t layer, const int32_t *routes,
                           const int32_t *sent, const int32_t *build, const int32_t *age,
                           void *hip_stream);

/* Diagnostics of the most recent relay: per-row alpha and beta (binary32,
 * beta = -INFINITY for an empty C) and the compacted rerouted row ids, one
 * ascending list per head at ids[h*n_q .. h*n_q + count_h), -1 after it
 * (formed from the relay's flags when asked for).  Each output may be NULL. */
rr_status rr_ledger_relay_stats(const rr_ledger *ledger, float *alpha, float *beta,
                                int32_t *ids, void *hip_stream);

/* Kernel timing for measurement.  Between rr_profile_start and
 * rr_profile_stop every kernel the library launches is bracketed by HIP
 * events recorded on its own stream.  rr_profile_stop waits for those events
 * and returns, per kernel kind, the summed duration in milliseconds and the
 * number of launches.  total_ms and launches are caller arrays of n_kinds
 * entries (each may be NULL); RR_KERNEL_KINDS entries are written, and
 * n_kinds < RR_KERNEL_KINDS with a non-NULL array returns RR_ERR_INVALID
 * without writing anything (profiling then stays on).  Process-wide; not for
 * concurrent use from several threads. */
typedef enum {
    RR_KERNEL_FULL = 0,     /* GEMM + TopK, full routing */
    RR_KERNEL_ANCHOR = 1,   /* GEMM + TopK + ledger build, every row */
    RR_KERNEL_REROUTE = 2,  /* GEMM + TopK + ledger build, compacted rows */
    RR_KERNEL_RESCORE = 3,  /* rescoring (dense tiles or gather), trigger, compaction counts, ages */
    RR_KERNEL_RELAY = 4,    /* one-pass relay: rescoring + trigger + GEMM + TopK + ledger build of the flagged rows */
    RR_KERNEL_POOL = 5,     /* chunk pooling */
    RR_KERNEL_EXPAND = 6,   /* token expansion */
    RR_KERNEL_ATTENTION = 7, /* sparse attention over routed chunks */
    RR_KERNEL_KINDS = 8
} rr_kernel_kind;

rr_status rr_profile_start(void);
rr_status rr_profile_stop(double *total_ms, int64_t *launches, int32_t n_kinds);

/* Exact selection (Eq. (2)) runs collection sweeps over a row's keys until
 * the row's candidate list holds exactly its top k+m (bisection on the score,
 * then on the chunk id of a tied score); the number of sweeps is capped above
 * what the bisections can need.  A row that still had not settled at the cap
 * would get an empty routed and near-miss set, and is counted here.
 * rr_unconverged_rows synchronises the current device and stores, in *count
 * (host memory), the number of such rows over every call on that device since
 * the library was loaded: 0 unless something is wrong.  A diagnostic, not for
 * the hot path. */
rr_status rr_unconverged_rows(uint64_t *count);

/* Test hook: caps the collection sweeps per route tile at `cap` for later
 * launches from this process (0 restores the default cap; the default always
 * suffices).  A lowered cap exists only to exercise rr_unconverged_rows. */
rr_status rr_set_sweep_cap(int32_t cap);

/* Number of bytes of ledger index storage (routes plus sentinels) for a
 * config: H_q * n_q * (k + m + r + n_sink + n_recent) * 4. */
size_t rr_ledger_index_bytes(const rr_config *cfg);

const char *rr_status_string(rr_status status);

/* Message of the calling thread's most recent failure ("" if none). */
const char *rr_last_error(void);

/* ------------------------------------------------------------------------
 * The steps either side of route maintenance.  Chunks are consecutive runs of
 * `chunk` tokens, the last one possibly shorter: n_chunks =
 * ceil(n_tokens / chunk), chunk j holds tokens j*chunk .. min((j+1)*chunk,
 * n_tokens) - 1.  All pointers are device memory; every call enqueues on the
 * given HIP stream (NULL: the default stream) and returns.
 * ---------------------------------------------------------------------- */

/* Chunk representations (Sec. 2.1: the router forms one representation per
 * chunk of tokens; here the mean of the chunk's token vectors).  X is
 * [n_heads, n_tokens, d] of dtype (rr_dtype), Xc receives [n_heads, n_chunks,
 * d] of the same dtype: each chunk's mean, summed in binary32 and rounded to
 * nearest even for bf16.  d a multiple of 8, at most 1024; chunk >= 1.
 * Returns RR_ERR_INVALID for bad sizes or NULL pointers. */
rr_status rr_pool_chunks(const void *X, int32_t n_heads, int32_t n_tokens, int32_t d, int32_t chunk,
                         int32_t dtype, void *Xc, void *hip_stream);

/* Token expansion (Sec. 2.1: selected chunks are expanded into token
 * indices).  routes is [rows, k] chunk ids (a ledger's or rr_full_route's
 * layout), tokens receives [rows, k*chunk] int32: route slot s fills columns
 * s*chunk .. s*chunk + chunk - 1 with its chunk's token ids ascending, -1
 * past the sequence's last token and for an empty (-1) or out-of-range slot.
 * Returns RR_ERR_INVALID for bad sizes or NULL pointers. */
rr_status rr_expand_tokens(const int32_t *routes, int64_t rows, int32_t k, int32_t chunk, int32_t n_tokens,
                           int32_t *tokens, void *hip_stream);

/* Sparse attention over routed chunks (Sec. 2.2 Eq. (3)): every query token t
 * of chunk i of head h attends, with one softmax scaled by `scale`, to the
 * tokens of the chunks in row h*n_chunks + i of routes; when causal, keys
 * after t are excluded (and routed chunks after i contribute nothing).  Slots
 * holding -1 or an id outside [0, n_chunks) are skipped; a query with no
 * admissible key gets a zero output.  Query head h reads key / value head
 * h / (n_heads / n_kv_heads).  Layouts: Q and O [n_heads, n_tokens, d], K and
 * V [n_kv_heads, n_tokens, d], bf16, row-major; routes [n_heads*n_chunks, k]
 * int32.  Scores and sums in binary32, the softmax weights rounded to bf16
 * for the value product, O rounded to nearest even.  Supported: bf16 with
 * d = 64 or 128, 1 <= k <= 256.  Returns RR_ERR_INVALID for bad sizes or NULL
 * pointers, RR_ERR_UNSUPPORTED for other dtypes or d. */
typedef struct {
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t n_tokens;
    int32_t d;
    int32_t chunk;      /* tokens per chunk */
    int32_t k;          /* route slots per row */
    int32_t causal;     /* 1: key token u is visible to query token t iff u <= t */
    int32_t dtype;      /* rr_dtype of Q, K, V and O (RR_BF16) */
    float scale;        /* softmax scale; 0: 1/sqrt(d) */
    int32_t reserved;   /* must be 0 */
} rr_attn_config;

rr_status rr_sparse_attention(const rr_attn_config *cfg, const void *Q, const void *K, const void *V,
                              const int32_t *routes, void *O, void *hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* ROUTERELAY_H */
