// Candidate rescoring, trigger and compaction bookkeeping for gfx950
// (RouteRelay, arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// Each row's candidates are its ledger slots: R (k slots), then the near-miss
// sentinels (m) and the random sentinels (r); -1 slots are empty.  Rescoring
// is a sampled product: only the (row, slot) pairs named by the ledger are
// scored, each as a dot product over d, with the key rows gathered straight
// from L2 (a head's key matrix is read by every workgroup of the head, and
// the workgroup-to-head map keeps a key head's workgroups on one XCD).
//
// A wave scores one row at a time: 16 candidates per round, 4 lanes per
// candidate, each lane reading 16-byte pieces so that one load instruction
// covers 64 contiguous bytes of 16 key rows; the loads of all rounds are in
// flight before the first product, and the next row's slot ids and query are
// already requested.  The 4 partial dots of a candidate are summed with two
// DPP quad permutations.  Wave reductions (DPP row shifts and row
// broadcasts) give the row's alpha = min over R, beta = max over C and its
// candidate counts; one lane per row then forms the refresh flag (C
// non-empty and beta + gamma >= alpha), writes the mask, alpha and beta, and
// sets age = layer - build layer on rows that keep their route.  Each
// workgroup stores its flagged-row and score-pair counts in its own slot of a
// per-workgroup table (no atomics); the reroute kernel turns the table into
// its per-head tile list and the call's totals.  No host synchronisation.
#include <math.h>


#include "rr_device.hpp"
#include "rr_internal.hpp"
#include "rr_rescore.hpp"

namespace rr {
namespace {

constexpr int kThreads = 64 * kRescoreWaves;

template <typename DT>
__device__ __forceinline__ float dot16(const u32x4_t &q, const u32x4_t &k, float acc);

template <>
__device__ __forceinline__ float dot16<float>(const u32x4_t &q, const u32x4_t &k, float acc)
{
    acc = fmaf(__uint_as_float(q.x), __uint_as_float(k.x), acc);
    acc = fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
    acc = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
    acc = fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
    return acc;
}

template <>
__device__ __forceinline__ float dot16<bf16_t>(const u32x4_t &q, const u32x4_t &k, float acc)
{
    // each 32-bit lane of the pieces is an rvalue copy before the cast (a
    // bit cast of a vector-element lvalue reads element 0 on this compiler)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t qa = q[j], ka = k[j];
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, qa), __builtin_bit_cast(bf16x2_t, ka), acc,
                                              false);
    }
    return acc;
}

// Sum over aligned groups of LPC lanes (4 or 8) with DPP permutations, no
// LDS round trip: two quad permutations, then the half-row mirror, which
// pairs each lane of one quad with a lane of the neighbouring quad.
template <int LPC>
__device__ __forceinline__ float group_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));  // lane ^ 1
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));  // lane ^ 2
    if (LPC == 8)
        x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));  // 7 - lane
    return x;
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_move(float fill, float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(x), CTRL, ROW_MASK, 0xF, false));
}

// Minimum / maximum over the 64 lanes of a wave, returned to every lane:
// shifts within each row of 16 lanes, then row broadcasts carry rows 0..2
// into lane 63, which is read back as a scalar.
template <bool MIN>
__device__ __forceinline__ float wave_extremum(float v)
{
    constexpr float id = MIN ? INFINITY : -INFINITY;
    auto op = [](float a, float b) { return MIN ? fminf(a, b) : fmaxf(a, b); };
    v = op(v, dpp_move<0x111, 0xF>(id, v));  // row_shr:1
    v = op(v, dpp_move<0x112, 0xF>(id, v));  // row_shr:2
    v = op(v, dpp_move<0x114, 0xF>(id, v));  // row_shr:4
    v = op(v, dpp_move<0x118, 0xF>(id, v));  // row_shr:8: lane 15 of a row holds the row
    v = op(v, dpp_move<0x142, 0xA>(id, v));  // row_bcast:15 into rows 1, 3
    v = op(v, dpp_move<0x143, 0xC>(id, v));  // row_bcast:31 into rows 2, 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// E groups of 64 slots per row; a block of kRescoreWaves waves scores
// rows_per_wave consecutive rows per wave.
template <typename DT, int D, int E>
__global__ __launch_bounds__(kThreads) void rescore_kernel(RescoreArgs a)
{
    constexpr int ROWB = D * (int)sizeof(DT);
    constexpr int LPC = (ROWB >= 16 * kRescoreLanesPerCand) ? kRescoreLanesPerCand : 4;  // lanes per candidate
    constexpr int CPR = 64 / LPC;         // candidates per round
    constexpr int CH = ROWB / (16 * LPC);  // 16-byte pieces per lane
    static_assert(CH >= 1 && ROWB % (16 * LPC) == 0, "row bytes must be a multiple of 16 lanes-per-candidate");
    constexpr int NR = 64 * E / CPR;      // rounds
    constexpr int NWG = kRescoreWaves;

    __shared__ unsigned long long s_pairs[NWG];
    __shared__ unsigned s_cnt[NWG];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int G = lane / LPC, pq = lane % LPC;
    int h, blk;
    tile_of_block(blockIdx.x, a.n_heads, a.n_kv_heads, a.blocks_per_head, h, blk);
    const int rpw = a.rows_per_wave, RB = NWG * rpw;
    const int i0 = blk * RB + w * rpw;  // this wave's rows: i0 .. i0 + rpw - 1
    const int nrows = max(0, min(rpw, a.n_q - i0));
    const int group = a.n_heads / a.n_kv_heads;
    const int c_sent = a.m + a.r + a.n_mand, c_led = a.k + c_sent;
    const int rounds = (c_led + CPR - 1) / CPR;
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * ROWB;
    const unsigned char *Qb = reinterpret_cast<const unsigned char *>(a.Q);
    const int64_t row0 = (int64_t)h * a.n_q + i0;

    auto load_ids = [&](int64_t row, int (&idr)[E]) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int slot = e * 64 + lane;
            int id = -1;
            if (slot < a.k)
                id = a.led_routes[row * a.k + slot];
            else if (slot < c_led)
                id = a.led_sent[row * c_sent + (slot - a.k)];
            idr[e] = id;
        }
    };
    auto load_q = [&](int64_t row, u32x4_t (&qv)[CH]) {
#pragma unroll
        for (int c = 0; c < CH; ++c) qv[c] = *reinterpret_cast<const u32x4_t *>(Qb + row * ROWB + (c * LPC + pq) * 16);
    };

    float my_a = INFINITY, my_b = -INFINITY;
    int my_nc = 0, my_ns = 0;
    int idr[E];
    u32x4_t qv[CH];
    if (nrows > 0) {
        load_ids(row0, idr);
        load_q(row0, qv);
    }
    for (int q = 0; q < nrows; ++q) {
        int idn[E];
        u32x4_t qn[CH];
        if (q + 1 < nrows) {
            load_ids(row0 + q + 1, idn);
            load_q(row0 + q + 1, qn);
        }
        int ids[NR];
        u32x4_t kv[NR][CH];
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int slot = u * CPR + G;
            ids[u] = -1;
            if (u < rounds) {  // wave-uniform: rounds past the ledger width load nothing
                ids[u] = __shfl(idr[(u * CPR) >> 6], slot & 63, 64);
                const unsigned char *kp = Kg + (int64_t)max(ids[u], 0) * ROWB;
#pragma unroll
                for (int c = 0; c < CH; ++c) kv[u][c] = *reinterpret_cast<const u32x4_t *>(kp + (c * LPC + pq) * 16);
            }
        }
        float amin = INFINITY, bmax = -INFINITY;
        int nc = 0, ns = 0;
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int slot = u * CPR + G;
            float part = 0.0f;
#pragma unroll
            for (int c = 0; c < CH; ++c) part = dot16<DT>(qv[c], kv[u][c], part);
            part = group_sum<LPC>(part);
            const bool inR = ids[u] >= 0 && slot < a.k, inC = ids[u] >= 0 && slot >= a.k;
            amin = inR ? fminf(amin, part) : amin;
            bmax = inC ? fmaxf(bmax, part) : bmax;
            nc += __popcll(__ballot(inR && pq == 0));
            ns += __popcll(__ballot(inC && pq == 0));
        }
        amin = wave_extremum<true>(amin);
        bmax = wave_extremum<false>(bmax);
        if (lane == q) {
            my_a = amin;
            my_b = bmax;
            my_nc = nc;
            my_ns = ns;
        }
        if (q + 1 < nrows) {
#pragma unroll
            for (int e = 0; e < E; ++e) idr[e] = idn[e];
#pragma unroll
            for (int c = 0; c < CH; ++c) qv[c] = qn[c];
        }
    }

    unsigned long long pairs_t = 0;
    unsigned cnt_t = 0;
    if (lane < nrows) {
        const int i = i0 + lane;
        const int64_t row = row0 + lane;
        const bool flag = relay_trigger(my_ns, my_a, my_b, a.gamma, a.gamma_rows, row, a.layer,
                                        a.min_reuse > 0 ? a.led_build[row] : 0, a.min_reuse);
        a.flags[row] = flag ? 1 : 0;
        if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
        a.alpha[row] = my_a;
        a.beta[row] = my_b;
        if (!flag) a.led_age[row] = a.layer - a.led_build[row];
        const int ni = a.causal ? min(i + 1, a.n_k) : a.n_k;
        pairs_t = (unsigned long long)(my_nc + my_ns + (flag ? ni : 0));
        cnt_t = flag ? 1u : 0u;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        pairs_t += (unsigned long long)__shfl_xor((long long)pairs_t, off, 64);
        cnt_t += (unsigned)__shfl_xor((int)cnt_t, off, 64);
    }
    if (lane == 0) {
        s_pairs[w] = pairs_t;
        s_cnt[w] = cnt_t;
    }
    __syncthreads();
    if (tid == 0) {
        unsigned long long P2 = 0;
        unsigned C = 0;
#pragma unroll
        for (int v = 0; v < NWG; ++v) {
            P2 += s_pairs[v];
            C += s_cnt[v];
        }
        const int slot = h * a.blocks_per_head + blk;  // head-major
        a.blk_pairs[slot] = (int64_t)P2;
        a.blk_count[slot] = (int32_t)C;
    }
}

template <typename DT, int D>
hipError_t launch_d(const RescoreArgs &a, hipStream_t stream)
{
    const int grid = a.n_heads * a.blocks_per_head;
    const int c = a.k + a.m + a.r + a.n_mand;
    if (c <= 64)
        hipLaunchKernelGGL((rescore_kernel<DT, D, 1>), dim3(grid), dim3(kThreads), 0, stream, a);
    else if (c <= 128)
        hipLaunchKernelGGL((rescore_kernel<DT, D, 2>), dim3(grid), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((rescore_kernel<DT, D, 4>), dim3(grid), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

void rescore_geometry(int64_t rows, int n_q, int n_k, RescoreGeometry &g)
{
    // dense tiles when the key range is short enough for the bitmaps and the
    // tiles fill at least half the chip: 128-row tiles from a tile per
    // compute unit, else 64-row tiles (measured at n_k = 512 with 128 tiles of
    // 128 rows: 64-row tiles 19.0 us, 128-row 22.3; at n_k = 1024 with 256:
    // 42 against 29); otherwise the gather
    const int64_t heads = rows / n_q;
    const int64_t large = heads * ((n_q + kDenseRowsLarge - 1) / kDenseRowsLarge);
    const int64_t small = heads * ((n_q + kDenseRowsSmall - 1) / kDenseRowsSmall);
    g.dense = n_k <= kRescoreDenseMaxKeys && (large >= kRescoreDenseFullTiles || small >= kRescoreDenseMinTiles);
    if (g.dense) {
        // tiles over the whole key range; a bitmap row holds two word pairs
        // per 64 keys of the padded range plus one, so that rows lie an odd
        // number of pairs apart and the 32 rows a wave reads together fall in
        // distinct LDS banks
        g.rows_per_wave = 0;
        g.rows_per_block = large >= kRescoreDenseFullTiles ? kDenseRowsLarge : kDenseRowsSmall;
        g.blocks_per_head = (n_q + g.rows_per_block - 1) / g.rows_per_block;
        g.bm_words = 2 * ((n_k + 63) / 64) + 1;
        return;
    }
    g.bm_words = 0;
    // rows per wave: about kRescoreBlocks workgroups in all, never more rows
    // per workgroup than a head has
    int64_t per = rows / ((int64_t)kRescoreBlocks * kRescoreWaves);
    int rpw = 1;
    while (rpw * 2 <= kRescoreMaxRowsPerWave && rpw * 2 <= per) rpw *= 2;
    while (rpw > 1 && (int64_t)kRescoreWaves * (rpw / 2) >= n_q) rpw /= 2;
    g.rows_per_wave = rpw;
    g.rows_per_block = kRescoreWaves * rpw;
    g.blocks_per_head = (n_q + g.rows_per_block - 1) / g.rows_per_block;
}

hipError_t launch_rescore(const RescoreArgs &a, int dtype, hipStream_t stream)
{
    if (a.dense) return launch_rescore_dense(a, dtype, stream);
    if (dtype == 0) {
        switch (a.d) {
        case 32: return launch_d<float, 32>(a, stream);
        case 64: return launch_d<float, 64>(a, stream);
        case 128: return launch_d<float, 128>(a, stream);
        default: break;
        }
    } else {
        switch (a.d) {
        case 32: return launch_d<bf16_t, 32>(a, stream);
        case 64: return launch_d<bf16_t, 64>(a, stream);
        case 128: return launch_d<bf16_t, 128>(a, stream);
        case 256: return launch_d<bf16_t, 256>(a, stream);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
