// Candidate rescoring, trigger and compaction bookkeeping for gfx950
// (RouteRelay, arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// Each row's candidates are its ledger slots: R (k slots), then the near-miss
// sentinels (m) and the random sentinels (r); -1 slots are empty.  A wave
// scores its rows one after another: one coalesced load brings all of a row's
// slot ids (lane j holds slot j), then 16 candidates per round -- 4 lanes
// share a candidate's key row, each reading 16-byte pieces so that one load
// instruction covers 64 contiguous bytes of 16 rows -- with the loads of all
// rounds in flight before any product is formed and the next row's ids and
// query already requested.  The 4 partial dots of a candidate are summed with
// two DPP quad permutations and the score goes to LDS.  A second phase gives
// each row to one lane, which forms alpha = min over R, beta = max over C and
// the refresh flag (C non-empty and beta + gamma >= alpha), and sets
// age = layer - build layer on rows that keep their route.
//
// Score-pair counts and per-head refresh counts go to device accumulators;
// the last workgroup to finish (ticket counter) turns the per-head counts
// into the reroute kernel's tile table (heads in XCD-major order, so each
// XCD's reroute workgroups find their tiles in one contiguous range),
// publishes the totals and zeroes the accumulators and the ticket for the
// next call.  No host synchronisation.
#include <math.h>

#include "rr_device.hpp"
#include "rr_internal.hpp"

namespace rr {
namespace {

template <typename DT>
__device__ __forceinline__ float dot16(const uint4 &q, const uint4 &k, float acc);

template <>
__device__ __forceinline__ float dot16<float>(const uint4 &q, const uint4 &k, float acc)
{
    acc = fmaf(__uint_as_float(q.x), __uint_as_float(k.x), acc);
    acc = fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
    acc = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
    acc = fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
    return acc;
}

template <>
__device__ __forceinline__ float dot16<bf16_t>(const uint4 &q, const uint4 &k, float acc)
{
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.x),
                                          __builtin_bit_cast(bf16x2_t, k.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.y),
                                          __builtin_bit_cast(bf16x2_t, k.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.z),
                                          __builtin_bit_cast(bf16x2_t, k.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, q.w),
                                          __builtin_bit_cast(bf16x2_t, k.w), acc, false);
    return acc;
}

// Sum over the 4 lanes of a quad (DPP quad permutations, no LDS round trip).
__device__ __forceinline__ float quad_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));  // lane ^ 1
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));  // lane ^ 2
    return x;
}

template <typename DT, int D, int E>
__global__ __launch_bounds__(256) void rescore_kernel(RescoreArgs a)
{
    constexpr int ROWB = D * (int)sizeof(DT);
    constexpr int CH = ROWB / 64;  // 16-byte pieces per lane (4 lanes per candidate)
    static_assert(CH >= 1 && ROWB % 64 == 0, "row bytes must be a multiple of 64");
    constexpr int NR = 4 * E;               // rounds of 16 candidates
    constexpr int RPW = kRescoreRows / 4;   // rows per wave
    constexpr int SC = 64 * E + 1;          // LDS score row stride

    __shared__ float sc[4][RPW][SC];
    __shared__ int s_ncand[4][RPW], s_nsent[4][RPW];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int G = lane >> 2, p = lane & 3;
    int h, blk;
    tile_of_block(blockIdx.x, a.n_heads, a.n_kv_heads, a.blocks_per_head, h, blk);
    const int i0 = blk * kRescoreRows + wave * RPW;
    const int group = a.n_heads / a.n_kv_heads;
    const int c_sent = a.m + a.r, c_led = a.k + c_sent;
    const int rounds = (c_led + 15) >> 4;
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * ROWB;
    const unsigned char *Qb = reinterpret_cast<const unsigned char *>(a.Q);
    const int nrows = min(RPW, a.n_q - i0);

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
    auto load_q = [&](int64_t row, uint4 (&qv)[CH]) {
#pragma unroll
        for (int c = 0; c < CH; ++c) qv[c] = *reinterpret_cast<const uint4 *>(Qb + row * ROWB + (c * 4 + p) * 16);
    };
    // Scores of one row (NR rounds, all loads issued before the first product)
    // into sc[wave][q][slot]; an empty R slot reads +inf and an empty sentinel
    // slot -inf, so neither can be the minimum over R or the maximum over C.
    auto score_row = [&](int q, const int (&idr)[E], const uint4 (&qv)[CH]) {
        int ids[NR];
        uint4 kv[NR][CH];
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int slot = u * 16 + G;
            ids[u] = (u < rounds) ? __shfl(idr[u >> 2], slot & 63, 64) : -1;
            if (ids[u] >= 0) {
                const unsigned char *kp = Kg + (int64_t)ids[u] * ROWB;
#pragma unroll
                for (int c = 0; c < CH; ++c) kv[u][c] = *reinterpret_cast<const uint4 *>(kp + (c * 4 + p) * 16);
            }
        }
        int ncand = 0, nsent = 0;
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int slot = u * 16 + G;
            float part = 0.0f;
            if (ids[u] >= 0) {
#pragma unroll
                for (int c = 0; c < CH; ++c) part = dot16<DT>(qv[c], kv[u][c], part);
            }
            part = quad_sum(part);
            if (p == 0 && u < rounds) sc[wave][q][slot] = (ids[u] >= 0) ? part : (slot < a.k ? INFINITY : -INFINITY);
            ncand += __popcll(__ballot(ids[u] >= 0 && p == 0));
            nsent += __popcll(__ballot(ids[u] >= 0 && p == 0 && slot >= a.k));
        }
        if (lane == 0) {
            s_ncand[wave][q] = ncand;
            s_nsent[wave][q] = nsent;
        }
    };

    int idr[E];
    uint4 qv[CH];
    if (nrows > 0) {
        load_ids((int64_t)h * a.n_q + i0, idr);
        load_q((int64_t)h * a.n_q + i0, qv);
    }
    for (int q = 0; q < nrows; ++q) {
        int idn[E];
        uint4 qn[CH];
        if (q + 1 < nrows) {
            load_ids((int64_t)h * a.n_q + i0 + q + 1, idn);
            load_q((int64_t)h * a.n_q + i0 + q + 1, qn);
        }
        score_row(q, idr, qv);
        if (q + 1 < nrows) {
#pragma unroll
            for (int e = 0; e < E; ++e) idr[e] = idn[e];
#pragma unroll
            for (int c = 0; c < CH; ++c) qv[c] = qn[c];
        }
    }
    __syncthreads();

    // One lane per row: alpha, beta, the trigger, age, counts.
    unsigned long long pairs_w = 0;
    unsigned cnt_w = 0;
    if (lane < nrows) {
        const int i = i0 + lane;
        const int64_t row = (int64_t)h * a.n_q + i;
        const float *rs = sc[wave][lane];
        float amin = INFINITY, bmax = -INFINITY;
        for (int slot = 0; slot < a.k; ++slot) amin = fminf(amin, rs[slot]);
        for (int slot = a.k; slot < c_led; ++slot) bmax = fmaxf(bmax, rs[slot]);
        const int ncand = s_ncand[wave][lane], nsent = s_nsent[wave][lane];
        const bool flag = nsent > 0 && (bmax + a.gamma >= amin);
        a.flags[row] = flag ? 1 : 0;
        if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
        a.alpha[row] = amin;
        a.beta[row] = bmax;
        if (!flag) a.led_age[row] = a.layer - a.led_build[row];
        const int ni = a.causal ? min(i + 1, a.n_k) : a.n_k;
        pairs_w = (unsigned long long)(ncand + (flag ? ni : 0));
        cnt_w = flag ? 1u : 0u;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        pairs_w += (unsigned long long)__shfl_xor((long long)pairs_w, off, 64);
        cnt_w += (unsigned)__shfl_xor((int)cnt_w, off, 64);
    }

    __shared__ unsigned long long s_pairs[4];
    __shared__ unsigned s_cnt[4];
    __shared__ int s_last;
    if (lane == 0) {
        s_pairs[wave] = pairs_w;
        s_cnt[wave] = cnt_w;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned long long P = s_pairs[0] + s_pairs[1] + s_pairs[2] + s_pairs[3];
        const unsigned C = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
        if (P) atomicAdd(a.acc_pairs, P);
        if (C) atomicAdd(&a.acc_count[h], C);
        __threadfence();
        const unsigned tk = atomicAdd(a.ticket, 1u);
        s_last = (tk == gridDim.x - 1) ? 1 : 0;
    }
    __syncthreads();
    if (s_last && threadIdx.x == 0) {
        __threadfence();
        const unsigned long long P = __hip_atomic_load(a.acc_pairs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int tr = a.reroute_tile_rows;
        int base = 0, total = 0;
        for (int j = 0; j < a.n_heads; ++j) {
            const int hd = head_at(j, a.n_heads, a.n_kv_heads);
            const unsigned c = __hip_atomic_load(&a.acc_count[hd], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.tile_base[j] = base;
            base += (int)((c + tr - 1) / tr);
            total += (int)c;
            a.acc_count[hd] = 0u;
        }
        a.tile_base[a.n_heads] = base;
        *a.stat_pairs = (int64_t)P;
        *a.stat_nrr = total;
        if (a.pairs_out) *a.pairs_out = (int64_t)P;
        if (a.nrr_out) *a.nrr_out = total;
        *a.acc_pairs = 0ull;
        *a.ticket = 0u;
    }
}

template <typename DT, int D>
hipError_t launch_d(const RescoreArgs &a, hipStream_t stream)
{
    const int grid = a.n_heads * a.blocks_per_head;
    const int c = a.k + a.m + a.r;
    if (c <= 64)
        hipLaunchKernelGGL((rescore_kernel<DT, D, 1>), dim3(grid), dim3(256), 0, stream, a);
    else if (c <= 128)
        hipLaunchKernelGGL((rescore_kernel<DT, D, 2>), dim3(grid), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((rescore_kernel<DT, D, 4>), dim3(grid), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_rescore(const RescoreArgs &a, int dtype, hipStream_t stream)
{
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
