// Candidate rescoring, trigger and compaction bookkeeping for gfx950
// (RouteRelay, arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// Each row's candidates are its ledger slots: R (k slots), then the near-miss
// sentinels (m) and the random sentinels (r); -1 slots are empty.  Rescoring
// is a sampled product: only the (row, slot) pairs named by the ledger are
// scored, each as a dot product over d.
//
// Gathering candidate key rows straight from L2 is bound by the vector L1's
// request rate (every 256-byte key row is a separate random access), so a
// workgroup instead stages its head's whole key matrix in LDS, one slice of
// the d range at a time: pass p holds bytes [16 P p, 16 P (p+1)) of every key
// row (P 16-byte pieces per key, P a power of two chosen so that n_k * P * 16
// bytes fit the LDS budget), together with the same slice of the block's query
// rows.  Lane j of a wave owns slot j (j + 64 e for the e-th group of 64 slots)
// of the wave's current row and accumulates its dot over the pass's pieces.
// The lanes of a wave read their pieces in a lane-rotated order (piece
// (u + lane) mod P at step u): key rows are P * 16 bytes apart, so the 8 lanes
// of an LDS access group read distinct 16-byte bank groups whatever the key
// ids are (for P >= 8).  The partial dots stay in registers across passes.
//
// After the last pass, wave reductions over the slot lanes give each row
// alpha = min over R, beta = max over C and its candidate count; one lane per
// row forms the refresh flag (C non-empty and beta + gamma >= alpha), writes
// the mask, alpha and beta, and sets age = layer - build layer on rows that
// keep their route.  Each workgroup stores its flagged-row and score-pair
// counts in its own slot of a per-workgroup table (no atomics); the reroute
// kernel turns the table into its per-head tile list and the call's totals.
// No host synchronisation.
#include <math.h>

#include "rr_device.hpp"
#include "rr_internal.hpp"

namespace rr {
namespace {

constexpr int kWaves = kRescoreWaves;  // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kStageUnroll = 8;  // staging loads in flight per thread

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

// E groups of 64 slots per row; each wave scores up to RPW rows of the block
// (the block holds rows_per_block = kWaves * rows_per_wave rows).
template <typename DT, int D, int E>
__global__ __launch_bounds__(kThreads) void rescore_kernel(RescoreArgs a)
{
    constexpr int ROWB = D * (int)sizeof(DT);
    constexpr int DP = ROWB / 16;        // 16-byte pieces per key row
    constexpr int RPW = kRescoreSlotRows / E;  // register budget: RPW * E partial dots per lane
    static_assert(ROWB % 16 == 0, "key rows are whole 16-byte pieces");

    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ unsigned long long s_pairs[kWaves];
    __shared__ unsigned s_cnt[kWaves];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int h, blk;
    tile_of_block(blockIdx.x, a.n_heads, a.n_kv_heads, a.blocks_per_head, h, blk);
    const int rpw = a.rows_per_wave;
    const int RB = kWaves * rpw;
    const int i0 = blk * RB;
    const int nrows = min(RB, a.n_q - i0);
    const int group = a.n_heads / a.n_kv_heads;
    const int c_sent = a.m + a.r, c_led = a.k + c_sent;
    const int P = a.pieces;  // pieces per key per pass (power of two, divides DP)
    const int npass = DP / P;
    const int64_t row0 = (int64_t)h * a.n_q + i0;

    u32x4_t *kb = reinterpret_cast<u32x4_t *>(smem);        // [n_k][P]
    u32x4_t *qb = kb + (int64_t)a.n_k * P;                     // [RB][P]
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * ROWB;
    const unsigned char *Qg = reinterpret_cast<const unsigned char *>(a.Q) + row0 * ROWB;

    // slot ids of this wave's rows (local row w + kWaves * q), lane j <-> slot j + 64 e
    int ids[RPW][E];
    float acc[RPW][E];
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
        const int lr = w + kWaves * q;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int slot = e * 64 + lane;
            int id = -1;
            if (q < rpw && lr < nrows) {
                const int64_t row = row0 + lr;
                if (slot < a.k)
                    id = a.led_routes[row * a.k + slot];
                else if (slot < c_led)
                    id = a.led_sent[row * c_sent + (slot - a.k)];
            }
            ids[q][e] = id;
            acc[q][e] = 0.0f;
        }
    }

    for (int ps = 0; ps < npass; ++ps) {
        if (ps > 0) __syncthreads();  // every wave is done with the previous slice
        // stage slice ps of the key rows and of the block's query rows
        const int nk = a.n_k * P, lp = __builtin_ctz(P);
        for (int t0 = tid; t0 < nk; t0 += kStageUnroll * kThreads) {
            u32x4_t v[kStageUnroll];
#pragma unroll
            for (int u = 0; u < kStageUnroll; ++u) {
                const int t = min(t0 + u * kThreads, nk - 1);  // clamped: the loads carry no branch
                const int key = t >> lp, pc = t & (P - 1);
                v[u] = *reinterpret_cast<const u32x4_t *>(Kg + (int64_t)key * ROWB + (ps * P + pc) * 16);
            }
#pragma unroll
            for (int u = 0; u < kStageUnroll; ++u)
                if (t0 + u * kThreads < nk) kb[t0 + u * kThreads] = v[u];
        }
        for (int t = tid; t < nrows * P; t += kThreads) {
            const int r = t >> lp, pc = t & (P - 1);
            qb[t] = *reinterpret_cast<const u32x4_t *>(Qg + (int64_t)r * ROWB + (ps * P + pc) * 16);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int lr = w + kWaves * q;
            if (q < rpw && lr < nrows) {
                const u32x4_t *qr = qb + lr * P;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const int id = ids[q][e];
                    if (id >= 0) {
                        const u32x4_t *kr = kb + (int64_t)id * P;
                        float s = acc[q][e];
                        for (int u = 0; u < P; ++u) {
                            const int pc = (u + lane) & (P - 1);
                            s = dot16<DT>(qr[pc], kr[pc], s);
                        }
                        acc[q][e] = s;
                    }
                }
            }
        }
    }
    // per row: alpha, beta and the candidate counts by wave reductions; lane q
    // keeps row q's values
    float my_a = INFINITY, my_b = -INFINITY;
    int my_nc = 0, my_ns = 0;
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
        const int lr = w + kWaves * q;
        if (q < rpw && lr < nrows) {
            float amin = INFINITY, bmax = -INFINITY;
            int nc = 0, ns = 0;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int slot = e * 64 + lane;
                const bool inR = ids[q][e] >= 0 && slot < a.k, inC = ids[q][e] >= 0 && slot >= a.k;
                amin = inR ? fminf(amin, acc[q][e]) : amin;
                bmax = inC ? fmaxf(bmax, acc[q][e]) : bmax;
                nc += __popcll(__ballot(inR));
                ns += __popcll(__ballot(inC));
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                amin = fminf(amin, __shfl_xor(amin, off, 64));
                bmax = fmaxf(bmax, __shfl_xor(bmax, off, 64));
            }
            if (lane == q) {
                my_a = amin;
                my_b = bmax;
                my_nc = nc;
                my_ns = ns;
            }
        }
    }

    // one lane per row: the trigger, outputs, age, counts
    unsigned long long pairs_t = 0;
    unsigned cnt_t = 0;
    {
        const int lr = w + kWaves * lane;
        if (lane < rpw && lr < nrows) {
            const int i = i0 + lr;
            const int64_t row = row0 + lr;
            const bool flag = my_ns > 0 && (my_b + a.gamma >= my_a);
            a.flags[row] = flag ? 1 : 0;
            if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
            a.alpha[row] = my_a;
            a.beta[row] = my_b;
            if (!flag) a.led_age[row] = a.layer - a.led_build[row];
            const int ni = a.causal ? min(i + 1, a.n_k) : a.n_k;
            pairs_t = (unsigned long long)(my_nc + my_ns + (flag ? ni : 0));
            cnt_t = flag ? 1u : 0u;
        }
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
        for (int v = 0; v < kWaves; ++v) {
            P2 += s_pairs[v];
            C += s_cnt[v];
        }
        const int slot = h * a.blocks_per_head + blk;  // head-major
        a.blk_pairs[slot] = (int64_t)P2;
        a.blk_count[slot] = (int32_t)C;
    }
}

template <typename DT, int D, int E>
hipError_t launch_e(const RescoreArgs &a, size_t lds, hipStream_t stream)
{
    const void *fn = reinterpret_cast<const void *>(&rescore_kernel<DT, D, E>);
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    const int grid = a.n_heads * a.blocks_per_head;
    hipLaunchKernelGGL((rescore_kernel<DT, D, E>), dim3(grid), dim3(kThreads), lds, stream, a);
    return hipGetLastError();
}

template <typename DT, int D>
hipError_t launch_d(const RescoreArgs &a, size_t lds, hipStream_t stream)
{
    const int c = a.k + a.m + a.r;
    if (c <= 64) return launch_e<DT, D, 1>(a, lds, stream);
    if (c <= 128) return launch_e<DT, D, 2>(a, lds, stream);
    return launch_e<DT, D, 4>(a, lds, stream);
}

}  // namespace

void rescore_geometry(int dtype, int d, int n_k, int64_t rows, int c, int n_q, RescoreGeometry &g)
{
    const int e = (dtype == 0) ? 4 : 2;
    const int dp = d * e / 16;
    // pieces per key per pass: the largest power of two (dividing dp) whose
    // key slice fits the staging budget; one piece at the longest key counts
    int p = 1;
    while (p * 2 <= dp && (int64_t)n_k * p * 2 * 16 <= kRescoreKeyBudget) p *= 2;
    g.pieces = p;
    const int groups = (c + 63) / 64;
    const int E = groups <= 1 ? 1 : (groups <= 2 ? 2 : 4);
    const int rpw_max = kRescoreSlotRows / E;
    // rows per wave: enough workgroups to give every compute unit two
    int64_t per = rows / (512 * kRescoreWaves);
    int rpw = 1;
    while (rpw * 2 <= rpw_max && rpw * 2 <= per) rpw *= 2;
    // a block never spans heads: no more rows than n_q (rounded to waves)
    while (rpw > 1 && (int64_t)kRescoreWaves * (rpw / 2) >= n_q) rpw /= 2;
    g.rows_per_wave = rpw;
    g.rows_per_block = kRescoreWaves * rpw;
    g.blocks_per_head = (n_q + g.rows_per_block - 1) / g.rows_per_block;
    g.lds_bytes = (size_t)n_k * p * 16 + (size_t)g.rows_per_block * p * 16;
}

hipError_t launch_rescore(const RescoreArgs &a, int dtype, size_t lds, hipStream_t stream)
{
    if (dtype == 0) {
        switch (a.d) {
        case 32: return launch_d<float, 32>(a, lds, stream);
        case 64: return launch_d<float, 64>(a, lds, stream);
        case 128: return launch_d<float, 128>(a, lds, stream);
        default: break;
        }
    } else {
        switch (a.d) {
        case 32: return launch_d<bf16_t, 32>(a, lds, stream);
        case 64: return launch_d<bf16_t, 64>(a, lds, stream);
        case 128: return launch_d<bf16_t, 128>(a, lds, stream);
        case 256: return launch_d<bf16_t, 256>(a, lds, stream);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
