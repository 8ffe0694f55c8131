// Candidate rescoring, trigger and compaction bookkeeping for gfx950
// (RouteRelay, arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// Each row's candidates are its ledger slots: R (k slots), then the near-miss
// sentinels (m) and the random sentinels (r); -1 slots are empty.  A wave
// works on one row at a time: one coalesced load brings all of the row's
// slot ids (lane j holds slot j), then the wave scores 16 candidates per
// round -- 4 lanes share a candidate's key row, each reading 16-byte pieces
// so that one load instruction covers 64 contiguous bytes of 16 rows -- with
// the loads of several rounds in flight before any product is formed, and the
// next row's ids and query already requested.  The 4 partial dots of a
// candidate are summed with two lane swaps.
//
// From the scores it forms alpha = min over R, beta = max over C and the
// refresh flag (C non-empty and beta + gamma >= alpha).  For a refreshed row
// it also records theta = the (k+m)-th best candidate score: the row has at
// least k+m chunks scoring >= theta, so theta bounds its new (k+m)-th score
// from below and seeds the reroute kernel's threshold.  Rows that keep their
// route get age = layer - build layer.
//
// Score-pair counts and per-head refresh counts go to device accumulators;
// the last workgroup to finish (ticket counter) turns the per-head counts
// into the reroute kernel's tile table, publishes the totals and zeroes the
// accumulators and the ticket for the next call.  No host synchronisation.
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

// Descending bitonic sort of E*64 floats; element e*64 + lane is v[e].
template <int E>
__device__ __forceinline__ void wave_sort_desc(float (&v)[E], int lane)
{
#pragma unroll
    for (int kk = 2; kk <= 64 * E; kk <<= 1) {
#pragma unroll
        for (int j = kk >> 1; j > 0; j >>= 1) {
            if (j >= 64) {
                const int je = j >> 6;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    if ((e & je) == 0) {
                        const int e2 = e | je;
                        const bool desc = (((e << 6) | lane) & kk) == 0;
                        const float x = v[e], y = v[e2];
                        v[e] = desc ? fmaxf(x, y) : fminf(x, y);
                        v[e2] = desc ? fminf(x, y) : fmaxf(x, y);
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const float p = __shfl_xor(v[e], j, 64);
                    const bool desc = (((e << 6) | lane) & kk) == 0;
                    const bool lower = (lane & j) == 0;
                    v[e] = (desc == lower) ? fmaxf(v[e], p) : fminf(v[e], p);
                }
            }
        }
    }
}

template <typename DT, int D, int E>
__global__ __launch_bounds__(256) void rescore_kernel(RescoreArgs a)
{
    constexpr int ROWB = D * (int)sizeof(DT);
    constexpr int CH = ROWB / 64;  // 16-byte pieces per lane (4 lanes per candidate)
    static_assert(CH >= 1 && ROWB % 64 == 0, "row bytes must be a multiple of 64");
    constexpr int RB = (16 / CH) < 4 ? ((16 / CH) < 1 ? 1 : 16 / CH) : 4;  // rounds per batch
    constexpr int NR = 4 * E;                                             // max rounds
    constexpr int RPW = kRescoreRows / 4;                                 // rows per wave

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int G = lane >> 2, p = lane & 3;
    int h, blk;
    tile_of_block(blockIdx.x, a.n_heads, a.n_kv_heads, a.blocks_per_head, h, blk);
    const int i0 = blk * kRescoreRows + wave * RPW;
    const int group = a.n_heads / a.n_kv_heads;
    const int c_sent = a.m + a.r, c_led = a.k + c_sent;
    const int rounds = (c_led + 15) >> 4;
    const int T = a.k + a.m;
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * ROWB;
    const unsigned char *Qb = reinterpret_cast<const unsigned char *>(a.Q);

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

    unsigned long long pairs_w = 0;
    unsigned cnt_w = 0;
    int idr[E], idn[E];
    uint4 qv[CH], qn[CH];
    const int nrows = min(RPW, a.n_q - i0);
    if (nrows > 0) {
        load_ids((int64_t)h * a.n_q + i0, idr);
        load_q((int64_t)h * a.n_q + i0, qv);
    }
    for (int q = 0; q < nrows; ++q) {
        const int i = i0 + q;
        const int64_t row = (int64_t)h * a.n_q + i;
        float sc[NR];
        // gathers of all rounds, RB rounds in flight at a time
#pragma unroll
        for (int u0 = 0; u0 < NR; u0 += RB) {
            uint4 kv[RB][CH];
            int ids[RB];
#pragma unroll
            for (int b = 0; b < RB; ++b) {
                const int u = u0 + b;
                const int slot = u * 16 + G;
                ids[b] = (u < rounds) ? __shfl(idr[u >> 2], slot & 63, 64) : -1;
                if (ids[b] >= 0) {
                    const unsigned char *kp = Kg + (int64_t)ids[b] * ROWB;
#pragma unroll
                    for (int c = 0; c < CH; ++c) kv[b][c] = *reinterpret_cast<const uint4 *>(kp + (c * 4 + p) * 16);
                }
            }
            if (u0 == 0 && q + 1 < nrows) {
                load_ids(row + 1, idn);
                load_q(row + 1, qn);
            }
#pragma unroll
            for (int b = 0; b < RB; ++b) {
                float part = 0.0f;
                if (ids[b] >= 0) {
#pragma unroll
                    for (int c = 0; c < CH; ++c) part = dot16<DT>(qv[c], kv[b][c], part);
                }
                part += __shfl_xor(part, 1, 64);
                part += __shfl_xor(part, 2, 64);
                sc[u0 + b] = (ids[b] >= 0) ? part : NAN;
            }
        }
        float amin = INFINITY, bmax = -INFINITY;
        int ncand = 0;
        bool has_c = false;
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int slot = u * 16 + G;
            const bool valid = (u < rounds) && !isnan(sc[u]);
            if (valid) {
                if (slot < a.k)
                    amin = fminf(amin, sc[u]);
                else
                    bmax = fmaxf(bmax, sc[u]);
            }
            const uint64_t mv = __ballot(valid && p == 0);
            const uint64_t mc = __ballot(valid && p == 0 && slot >= a.k);
            ncand += __popcll(mv);
            has_c |= (mc != 0ull);
        }
#pragma unroll
        for (int off = 4; off < 64; off <<= 1) {
            amin = fminf(amin, __shfl_xor(amin, off, 64));
            bmax = fmaxf(bmax, __shfl_xor(bmax, off, 64));
        }
        const bool flag = has_c && (bmax + a.gamma >= amin);
        float theta = -INFINITY;
        if (flag) {
            // one score per lane (slot e*64 + lane), then the (k+m)-th best
            float v[E];
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int src = 4 * (lane & 15);
                float x = NAN;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const float y = __shfl(sc[4 * e + b], src, 64);
                    x = ((lane >> 4) == b) ? y : x;
                }
                v[e] = (idr[e] >= 0 && !isnan(x)) ? x : -INFINITY;
            }
            wave_sort_desc<E>(v, lane);
            if (ncand >= T) {
                float t = -INFINITY;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    if (((T - 1) >> 6) == e) t = v[e];
                theta = __shfl(t, (T - 1) & 63, 64);
            }
        }
        if (lane == 0) {
            a.flags[row] = flag ? 1 : 0;
            if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
            a.alpha[row] = amin;
            a.beta[row] = bmax;
            a.theta[row] = theta;
            if (!flag) a.led_age[row] = a.layer - a.led_build[row];
            const int ni = a.causal ? min(i + 1, a.n_k) : a.n_k;
            pairs_w += (unsigned long long)(ncand + (flag ? ni : 0));
            cnt_w += flag ? 1u : 0u;
        }
        if (q + 1 < nrows) {
#pragma unroll
            for (int e = 0; e < E; ++e) idr[e] = idn[e];
#pragma unroll
            for (int c = 0; c < CH; ++c) qv[c] = qn[c];
        }
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
        for (int hd = 0; hd < a.n_heads; ++hd) {
            const unsigned c = __hip_atomic_load(&a.acc_count[hd], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.tile_base[hd] = base;
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
