// Dense candidate rescoring for key heads of up to 2048 chunks (RouteRelay,
// arXiv 2609.07306, Sec. 3.2 Eq. (5)-(8); Sec. 4.1-4.2).
//
// The sampled product of Eq. (5) names at most k + m + r keys per row, but
// with n_k <= 2048 the candidates cover a few percent of a head's keys, and
// on matrix cores the full product of a 64- or 128-row tile with all of its head's
// keys costs less than gathering the candidate key rows one by one: the key
// head streams once per tile through LDS (the routing sweep's staging), the
// MFMAs produce every score, and the epilogue keeps a score only where the
// row's ledger names the key.  Each row's ledger is turned into two bitmaps
// over the key range (routed set R, candidate set C = near-miss + random
// sentinels); per stage a lane reads the words of its 16 keys and folds
//   alpha = min over R,  beta = max over C
// with bit-select (a masked-out score becomes +inf for the minimum, -inf for
// the maximum).  The scores are the ones the routing kernel computes (same
// fragments, same MFMA order), so a route's score at rescoring is bitwise the
// routing score when Q and K are unchanged.
//
// Row outputs and the per-workgroup tables match the gather kernel's: the
// refresh flag (C non-empty and beta + gamma >= alpha), mask, alpha, beta,
// the age of rows that keep their route, and per-tile flagged-row and
// score-pair counts (score pairs follow the method's accounting: the ledger's
// candidates, plus n_i for each refreshed row).

#include <algorithm>

#include "rr_rescore.hpp"
#include "rr_route_impl.hpp"

namespace rr {
namespace {

using route_detail::RT;

// Tiles of 32 * NW rows (NW = 4 or 2 row blocks); waves = row blocks x 2
// key splits.
template <typename DT, int D, int NW>
using DenseRT = RT<DT, D, NW, 2, 2, 64, 32>;
// Tiles whose key fragments take at most 256 bytes per row have the
// registers for the kept scores of the threshold step as well.
template <typename DT, int D>
constexpr bool kDenseSeeds = sizeof(DT) * D <= 256;

// SEED: the epilogue also keeps, per register slot, the top two scores of
// the valid keys passing through it (the routing kernel's threshold sweep),
// from which each row's bound of its (k+m)-th score and its maximum follow.
template <bool SEED>
struct DenseEpi {
    float amin, bmax;
    int sbase;         // first key of the lane's segment
    const uint2 *bmr;  // this lane's row: (R word, C word) per 32 keys
    int nrow;          // SEED: valid keys of the lane's row (0: padding row)
    float top[SEED ? 16 : 1][2];
    uint2 wnext;       // this stage's words, read a stage ahead (set to stage 0's
                       // before the sweep; the row's bitmap has a word past the
                       // last stage's)

    template <class F>
    __device__ __forceinline__ void step(int st, const f32x16_t &acc, f32x16_t &next, const F &fq, const F &fk,
                                         bool full)
    {
        const int k0 = sbase + 16 * st;  // this lane's keys: k0 .. k0 + 15 (k0 % 16 == 0)
        const uint2 wv = wnext;
        wnext = bmr[(k0 + 16) >> 5];
        next = route_detail::tile_product(fq, fk);
        const uint32_t sh = (uint32_t)(k0 & 16);
        const uint32_t mr = wv.x >> sh, mc = wv.y >> sh;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const uint32_t xb = __float_as_uint(acc[i]);
            // all-ones where key k0 + i is in the set, else zero
            const uint32_t nr = (uint32_t)((int32_t)(mr << (31 - i)) >> 31);
            const uint32_t nc = (uint32_t)((int32_t)(mc << (31 - i)) >> 31);
            amin = fminf(amin, __uint_as_float((xb & nr) | (0x7F800000u & ~nr)));  // +inf when out
            bmax = fmaxf(bmax, __uint_as_float((xb & nc) | (0xFF800000u & ~nc)));  // -inf when out
        }
        if constexpr (SEED) {
            if (full) {
#pragma unroll
                for (int i = 0; i < 16; ++i) route_detail::top_insert<2>(top[i], acc[i]);
            } else {
                const int vlim = nrow - k0;  // keys k0 + i are valid for i < vlim
#pragma unroll
                for (int i = 0; i < 16; ++i) route_detail::top_insert<2>(top[i], (i < vlim) ? acc[i] : -INFINITY);
            }
        }
        route_detail::interleave_mfma<F::NS, (16 * (SEED ? 8 : 6) + F::NS - 1) / F::NS>();
    }
};

template <typename DT, int D, int NW>
__global__ __launch_bounds__(128 * NW) void rescore_dense_kernel(RescoreArgs a)
{
    using C = DenseRT<DT, D, NW>;
    static_assert(C::NT == 128 * NW, "launch bounds of the tile shape");
    constexpr bool SEED = kDenseSeeds<DT, D>;
    constexpr int BM = C::BM, NT = C::NT, KS = 2;
    constexpr int NWB = (BM + 63) / 64;  // waves holding one lane per row
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *bt = smem;                                     // [2][KS][32][BSTR] key tiles
    uint2 *bm = reinterpret_cast<uint2 *>(smem + 2 * C::ST);      // [BM][bm_words] (R word, C word) pairs
    __shared__ int32_t row_n[BM], s_nc[BM], s_ns[BM];
    __shared__ float s_amin[KS][BM], s_bmax[KS][BM], s_b1[BM], s_rmx[BM];
    __shared__ unsigned long long s_pairs[NWB];
    __shared__ unsigned s_cnt[NWB];

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
    const int rb = w % NW, p = w / NW;
    const int nwd = a.bm_words;
    int h, t;
    tile_of_block(blockIdx.x, a.n_heads, a.n_kv_heads, a.blocks_per_head, h, t);
    const int i0 = t * BM;
    const int64_t g0 = (int64_t)h * a.n_q + i0;  // first row of the tile
    const int c_sent = a.m + a.r + a.n_mand, c_led = a.k + c_sent;

    // the tile's longest valid key range (tiles always hold a row), and the
    // first two key stages, the query fragments and the ledger rows are all
    // requested before the bitmap set-up, whose barriers order LDS only
    const int ncols = a.causal ? min(min(i0 + BM, a.n_q), a.n_k) : a.n_k;
    const int nb = __builtin_amdgcn_readfirstlane((ncols + 32 * KS - 1) / (32 * KS));
    const int seg = 16 * nb;
    const unsigned char *Kg = reinterpret_cast<const unsigned char *>(a.K) +
                              (int64_t)(h / (a.n_heads / a.n_kv_heads)) * a.n_k * C::ROWB;
    // double-buffered key fragments where a second set fits in registers
    constexpr bool kDb = sizeof(DT) * D <= 256;
    u32x4_t breg[2][C::PER_T];
    if constexpr (kDb) route_detail::sweep_db_first<C>(breg, Kg, a.n_k, seg, nb, tid);
    const int myrow = 32 * rb + l32;
    const int myseg = 2 * p + hh;
    const int mi = i0 + myrow;
    const int nrow = (mi < a.n_q) ? (a.causal ? min(mi + 1, a.n_k) : a.n_k) : 0;
    // stages whose keys (up to (2p+1)*seg + 16 st + 15) are valid for every
    // row of the wave (the kept scores mask the others)
    int full_stages = nb;
    if constexpr (SEED) {
        int minn = (mi < a.n_q) ? nrow : INT_MAX;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) minn = min(minn, __shfl_xor(minn, off, 64));
        const int slack = minn - (2 * p + 1) * seg - 16;
        full_stages = __builtin_amdgcn_readfirstlane(
            (minn == INT_MAX) ? nb : (slack < 0 ? 0 : min(nb, slack / 16 + 1)));
    }
    Frag<DT, D> fq;
    if (i0 + myrow < a.n_q)
        fq.load(reinterpret_cast<const DT *>(a.Q) + (g0 + myrow) * D, hh);
    else
        fq.zero();

    // ledger rows -> bitmaps.  Wave w takes rows w, w + 8, ... (RPW rows),
    // lane = slot.  Every lane loads (rows past n_q and slots past the ledger
    // read the tile's first row and are masked), so the loads carry no
    // branches; the first chunk's loads are issued before the bitmaps are
    // cleared, and the set-up barriers order LDS only, so the query and
    // ledger loads are in flight together.  The counts are of the ledger's
    // filled slots.
    constexpr int RPW = BM / C::NWV;
    auto load_chunk = [&](int s0, int (&id)[RPW]) {
        // the lane's column of the ledger (routes or sentinels) and its row
        // stride, formed once, so the unrolled loads need no kernel argument
        const int slot = s0 + lane;
        const bool inr = slot < a.k, live = slot < c_led;
        const int32_t *col = inr ? a.led_routes + slot : (live ? a.led_sent + (slot - a.k) : a.led_routes);
        const int64_t stride = inr ? a.k : (live ? c_sent : a.k);
        const int nrow = min(BM, a.n_q - i0);  // rows of the tile
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int r = w + q * C::NWV;
            const bool ok = live && r < nrow;
            const int v = col[(g0 + (ok ? r : 0)) * stride];
            id[q] = ok ? v : -1;
        }
    };
    int id[RPW];
    load_chunk(0, id);

    for (int j = tid; j < BM * nwd; j += NT) bm[j] = make_uint2(0u, 0u);
    if (tid < BM) {
        const int i = i0 + tid;
        row_n[tid] = (i < a.n_q) ? (a.causal ? min(i + 1, a.n_k) : a.n_k) : 0;
    }
    lds_barrier();

    int nc[RPW], ns[RPW];
#pragma unroll
    for (int q = 0; q < RPW; ++q) nc[q] = ns[q] = 0;
    uint32_t *bw = reinterpret_cast<uint32_t *>(bm);
    for (int s0 = 0; s0 < c_led; s0 += 64) {
        if (s0 > 0) load_chunk(s0, id);
        const bool inr = s0 + lane < a.k;
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int r = w + q * C::NWV;
            const bool ok = id[q] >= 0 && id[q] < a.n_k;  // ledger ids lie in [0, n_i); -1 is an empty slot
            // word (id >> 5) of the row: .x holds R, .y holds C
            if (ok) atomicOr(&bw[2 * (r * nwd + (id[q] >> 5)) + (inr ? 0 : 1)], 1u << (id[q] & 31));
            nc[q] += __popcll(__ballot(ok && inr));
            ns[q] += __popcll(__ballot(ok && !inr));
        }
    }
    if (lane == 0) {
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int r = w + q * C::NWV;
            s_nc[r] = nc[q];
            s_ns[r] = ns[q];
        }
    }
    lds_barrier();

    DenseEpi<SEED> epi;
    epi.amin = INFINITY;
    epi.bmax = -INFINITY;
    epi.sbase = myseg * seg;
    epi.bmr = bm + myrow * nwd;
    epi.wnext = epi.bmr[epi.sbase >> 5];
    epi.nrow = nrow;
    if constexpr (SEED) {
#pragma unroll
        for (int i = 0; i < 16; ++i) epi.top[i][0] = epi.top[i][1] = -INFINITY;
    }
    if constexpr (kDb)
        route_detail::sweep_keys_db<DT, D, C>(fq, Kg, a.n_k, seg, nb, full_stages, tid, p, hh, l32, bt, breg, epi);
    else
        route_detail::sweep_keys<DT, D, C>(fq, Kg, a.n_k, seg, nb, full_stages, tid, p, hh, l32, bt, epi);

    // the row's four lanes: halves hh of a wave, then the key splits p
    float amin = fminf(epi.amin, __shfl_xor(epi.amin, 32, 64));
    float bmax = fmaxf(epi.bmax, __shfl_xor(epi.bmax, 32, 64));
    if (hh == 0) {
        s_amin[p][myrow] = amin;
        s_bmax[p][myrow] = bmax;
    }
    __syncthreads();  // (also: every wave is done with the key tiles and bitmaps)
    if constexpr (SEED) {
        // the routing kernel's threshold step on the same scores: kept sets
        // -> bound of the (k+m)-th score and the row maximum
        float *us = reinterpret_cast<float *>(smem);
        route_detail::store_kept<C, 2>(us, myrow, myseg, epi.top);
        __syncthreads();
        route_detail::bound_of_kept<C>(us, tid, a.k + a.m, s_b1, s_rmx);
        __syncthreads();
    }

    unsigned long long pairs_t = 0;
    unsigned cnt_t = 0;
    if (tid < BM && i0 + tid < a.n_q) {
        const int64_t row = g0 + tid;
        const float al = fminf(s_amin[0][tid], s_amin[1][tid]);
        const float be = fmaxf(s_bmax[0][tid], s_bmax[1][tid]);
        const int nc = s_nc[tid], ns = s_ns[tid];
        const bool flag = relay_trigger(ns, al, be, a.gamma, a.gamma_rows, row, a.layer,
                                        a.min_reuse > 0 ? a.led_build[row] : 0, a.min_reuse);
        a.flags[row] = flag ? 1 : 0;
        if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
        a.alpha[row] = al;
        a.beta[row] = be;
        if (!flag) a.led_age[row] = a.layer - a.led_build[row];
        if (SEED && a.seed_bound) {
            a.seed_bound[row] = s_b1[tid];
            a.seed_rmax[row] = s_rmx[tid];
        }
        pairs_t = (unsigned long long)(nc + ns + (flag ? row_n[tid] : 0));
        cnt_t = flag ? 1u : 0u;
    }
    if (tid < 64 * NWB) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            pairs_t += (unsigned long long)__shfl_xor((long long)pairs_t, off, 64);
            cnt_t += (unsigned)__shfl_xor((int)cnt_t, off, 64);
        }
        if (lane == 0) {
            s_pairs[w] = pairs_t;
            s_cnt[w] = cnt_t;
        }
    }
    __syncthreads();
    if (tid == 0) {
        const int slot = h * a.blocks_per_head + t;  // head-major
        unsigned long long P2 = 0;
        unsigned Cn = 0;
#pragma unroll
        for (int v = 0; v < NWB; ++v) {
            P2 += s_pairs[v];
            Cn += s_cnt[v];
        }
        a.blk_pairs[slot] = (int64_t)P2;
        a.blk_count[slot] = (int32_t)Cn;
    }
}

template <typename DT, int D, int NW>
hipError_t launch_n(const RescoreArgs &a, hipStream_t stream)
{
    using C = DenseRT<DT, D, NW>;
    size_t lds = (size_t)2 * C::ST + (size_t)C::BM * a.bm_words * sizeof(uint2);
    if (kDenseSeeds<DT, D>) lds = std::max(lds, (size_t)C::BM * C::UST * sizeof(float));  // the kept scores
    const void *fn = reinterpret_cast<const void *>(&rescore_dense_kernel<DT, D, NW>);
    static LdsLimit seen;
    const hipError_t e = raise_lds_limit(fn, lds, seen);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((rescore_dense_kernel<DT, D, NW>), dim3(a.n_heads * a.blocks_per_head), dim3(C::NT), lds,
                       stream, a);
    return hipGetLastError();
}

template <typename DT, int D>
hipError_t launch_d(const RescoreArgs &a, hipStream_t stream)
{
    static_assert(DenseRT<DT, D, 4>::BM == kDenseRowsLarge && DenseRT<DT, D, 2>::BM == kDenseRowsSmall,
                  "dense tile heights");
    if (a.rows_per_block == kDenseRowsSmall) return launch_n<DT, D, 2>(a, stream);
    if (a.rows_per_block == kDenseRowsLarge) return launch_n<DT, D, 4>(a, stream);
    return hipErrorInvalidValue;
}

}  // namespace

bool rescore_dense_seeds(int dtype, int d)
{
    return (dtype == 0 ? kDenseSeeds<float, 64> : kDenseSeeds<bf16_t, 128>) && (dtype == 0 ? 4 : 2) * d <= 256;
}

hipError_t launch_rescore_dense(const RescoreArgs &a, int dtype, hipStream_t stream)
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
