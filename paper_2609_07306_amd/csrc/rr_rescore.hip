// Candidate rescoring, trigger and compaction bookkeeping for gfx950
// (RouteRelay, arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// Each row's candidates are its ledger slots: R (k slots), then the near-miss
// sentinels (m) and the random sentinels (r); -1 slots are empty.  A wave
// scores 16 candidates at a time: 4 lanes share a candidate's key row, each
// reading 16-byte pieces so that every load instruction covers 64 contiguous
// bytes of 16 rows, and the 4 partial dots are summed with two lane swaps.
// From the scores it forms alpha = min over R, beta = max over C and the
// refresh flag (C non-empty and beta + gamma >= alpha), and the lower bound
// theta = min over R and the near-miss slots that seeds the reroute
// threshold (those k+m chunks all score at least theta, so the row's
// (k+m)-th score is >= theta).  Rows that keep their route get
// age = layer - build layer.
//
// Workgroups cover 64 rows of one head.  Their score-pair counts and per-head
// flag counts go to device accumulators with atomics; the last workgroup to
// finish (a ticket counter) turns the per-head counts into the tile table of
// the reroute kernel, publishes the totals and zeroes the accumulators and
// the ticket for the next call.  Nothing here needs a host synchronisation.
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

template <typename DT, int D>
__global__ __launch_bounds__(256) void rescore_kernel(RescoreArgs a)
{
    constexpr int ROWB = D * (int)sizeof(DT);
    constexpr int CH = ROWB / 64;  // 16-byte pieces per lane (4 lanes per candidate)
    static_assert(CH >= 1 && ROWB % 64 == 0, "row bytes must be a multiple of 64");
    constexpr int RPW = kRescoreRows / 4;  // rows per wave

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int G = lane >> 2, p = lane & 3;
    const int h = blockIdx.x / a.blocks_per_head;
    const int i0 = (blockIdx.x % a.blocks_per_head) * kRescoreRows;
    const int group = a.n_heads / a.n_kv_heads;
    const int c_sent = a.m + a.r, c_led = a.k + c_sent;
    const int rounds = (c_led + 15) >> 4;
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * ROWB;

    unsigned long long pairs_w = 0;
    unsigned cnt_w = 0;
    for (int q = 0; q < RPW; ++q) {
        const int i = i0 + wave * RPW + q;
        if (i >= a.n_q) break;
        const int64_t row = (int64_t)h * a.n_q + i;
        const unsigned char *qp = reinterpret_cast<const unsigned char *>(a.Q) + row * ROWB;
        uint4 qv[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) qv[c] = *reinterpret_cast<const uint4 *>(qp + (c * 4 + p) * 16);

        float amin = INFINITY, bmax = -INFINITY, nmin = INFINITY;
        int ncand = 0;
        bool has_c = false;
        for (int u = 0; u < rounds; ++u) {
            const int slot = u * 16 + G;
            int id = -1;
            if (slot < a.k)
                id = a.led_routes[row * a.k + slot];
            else if (slot < c_led)
                id = a.led_sent[row * c_sent + (slot - a.k)];
            float part = 0.0f;
            if (id >= 0) {
                const unsigned char *kp = Kg + (int64_t)id * ROWB;
#pragma unroll
                for (int c = 0; c < CH; ++c)
                    part = dot16<DT>(qv[c], *reinterpret_cast<const uint4 *>(kp + (c * 4 + p) * 16), part);
            }
            part += __shfl_xor(part, 1, 64);
            part += __shfl_xor(part, 2, 64);
            if (id >= 0) {
                if (slot < a.k) {
                    amin = fminf(amin, part);
                } else {
                    bmax = fmaxf(bmax, part);
                    if (slot < a.k + a.m) nmin = fminf(nmin, part);
                }
            }
            const uint64_t mv = __ballot(id >= 0 && p == 0);
            const uint64_t mc = __ballot(id >= 0 && p == 0 && slot >= a.k);
            ncand += __popcll(mv);
            has_c |= (mc != 0ull);
        }
#pragma unroll
        for (int off = 4; off < 64; off <<= 1) {
            amin = fminf(amin, __shfl_xor(amin, off, 64));
            bmax = fmaxf(bmax, __shfl_xor(bmax, off, 64));
            nmin = fminf(nmin, __shfl_xor(nmin, off, 64));
        }
        const bool flag = has_c && (bmax + a.gamma >= amin);
        if (lane == 0) {
            a.flags[row] = flag ? 1 : 0;
            if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
            a.alpha[row] = amin;
            a.beta[row] = bmax;
            a.theta[row] = fminf(amin, nmin);
            if (!flag) a.led_age[row] = a.layer - a.led_build[row];
            const int ni = a.causal ? min(i + 1, a.n_k) : a.n_k;
            pairs_w += (unsigned long long)(ncand + (flag ? ni : 0));
            cnt_w += flag ? 1u : 0u;
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
        int base = 0, total = 0;
        for (int hd = 0; hd < a.n_heads; ++hd) {
            const unsigned c = __hip_atomic_load(&a.acc_count[hd], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.tile_base[hd] = base;
            base += (int)((c + kTileRows - 1) / kTileRows);
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
hipError_t launch_t(const RescoreArgs &a, hipStream_t stream)
{
    const int grid = a.n_heads * a.blocks_per_head;
    hipLaunchKernelGGL((rescore_kernel<DT, D>), dim3(grid), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_rescore(const RescoreArgs &a, int dtype, hipStream_t stream)
{
    if (dtype == 0) {
        switch (a.d) {
        case 32: return launch_t<float, 32>(a, stream);
        case 64: return launch_t<float, 64>(a, stream);
        case 128: return launch_t<float, 128>(a, stream);
        default: break;
        }
    } else {
        switch (a.d) {
        case 32: return launch_t<bf16_t, 32>(a, stream);
        case 64: return launch_t<bf16_t, 64>(a, stream);
        case 128: return launch_t<bf16_t, 128>(a, stream);
        case 256: return launch_t<bf16_t, 256>(a, stream);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
