// Row-wise GEMM + TopK routing for gfx950 (RouteRelay, arXiv 2609.07306).
//
// One kernel serves three callers:
//   MODE_FULL    -- full routing of every row, Eq. (1)-(2) (the baseline);
//   MODE_ANCHOR  -- full routing plus the ledger build of Sec. 3.1: the
//                   chunks ranked k+1..k+m become near-miss sentinels and r
//                   random sentinels are drawn from what is left;
//   MODE_REROUTE -- the same for the rows a relay layer flagged (Sec. 3.2,
//                   row-selective refresh of Sec. 4.2), read per head from
//                   the flag array in ascending row order.
//
// A workgroup is one wave and owns a tile of 32 query rows of one head.  It
// streams the head's key chunks 32 at a time through a 32x32 MFMA tile
// (v_mfma_f32_32x32x16_bf16 or v_mfma_f32_32x32x2_f32); the score matrix is
// never stored.  Selecting T = k + m chunks per row works in two sweeps:
//   1. a threshold: each lane keeps its top-t scores of each of its 16 rows
//      (t = 2 for T <= 64, 4 for T <= 128).  The ceil(T/t)-th largest
//      lane-local t-th score over the 32 lanes of a row bounds the row's T-th
//      score from below (at least t * ceil(T/t) >= T scores reach it).
//      Reroute tiles skip this sweep and start from the bound the rescoring
//      kernel derived from the ledger's own candidates (minus a small margin).
//   2. a collection: scores at or above the threshold are appended, in chunk
//      id order, to a per-row LDS list.  A list that came out short of
//      min(T, n_i) (a seeded bound that was too high) is redone with the
//      sweep-1 bound; a list that overflowed is redone with the T-th best of
//      its first entries as the (score, id) threshold.  Both cases only raise
//      correctness work, never change the result.
// The final order statistics come from a bitonic sort of the row's list on
// 64-bit (score, id) keys; a second pass over the id-ordered list writes R
// and the near-miss set already sorted by chunk id.
#include <limits.h>
#include <math.h>

#include "rr_device.hpp"
#include "rr_internal.hpp"

namespace rr {
namespace {

constexpr int kMaxFixIters = 40;  // bound on threshold repairs per tile

// Descending bitonic sort of one float per lane across each 32-lane half.
__device__ __forceinline__ float sort32_desc(float x, int l32)
{
#pragma unroll
    for (int kk = 2; kk <= 32; kk <<= 1) {
#pragma unroll
        for (int j = kk >> 1; j > 0; j >>= 1) {
            float p = __shfl_xor(x, j, 64);
            bool desc = (l32 & kk) == 0;
            bool lower = (l32 & j) == 0;
            x = (desc == lower) ? fmaxf(x, p) : fminf(x, p);
        }
    }
    return x;
}

// Descending bitonic sort of E*64 keys; element e*64 + lane lives in key[e].
template <int E>
__device__ __forceinline__ void sort_keys_desc(uint64_t (&key)[E], int lane)
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
                        const uint64_t x = key[e], y = key[e2];
                        const bool sw = desc ? (x < y) : (x > y);
                        key[e] = sw ? y : x;
                        key[e2] = sw ? x : y;
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const uint64_t p = shfl_xor_u64(key[e], j);
                    const bool desc = (((e << 6) | lane) & kk) == 0;
                    const bool lower = (lane & j) == 0;
                    const uint64_t mx = key[e] > p ? key[e] : p;
                    const uint64_t mn = key[e] > p ? p : key[e];
                    key[e] = (desc == lower) ? mx : mn;
                }
            }
        }
    }
}

template <int E>
__device__ __forceinline__ uint64_t key_at(const uint64_t (&key)[E], int p)
{
    uint64_t v = 0;
#pragma unroll
    for (int e = 0; e < E; ++e)
        if ((p >> 6) == e) v = key[e];
    return shfl_u64(v, p & 63);
}

// Keys of rank min(kk, c) and min(TT, c) (1-based) among the c entries of an
// LDS list.  Called by the whole wave.
template <int CAP>
__device__ void select_bounds(const float *rs, const int32_t *ri, int c, int kk, int TT, int lane,
                              uint64_t &key_k, uint64_t &key_T)
{
    constexpr int E = CAP / 64;
    uint64_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = (e << 6) + lane;
        key[e] = idx < c ? rank_key(rs[idx], ri[idx]) : 0ull;
    }
    sort_keys_desc<E>(key, lane);
    const int pk = min(kk, c) - 1, pT = min(TT, c) - 1;
    key_k = pk >= 0 ? key_at<E>(key, pk) : ~0ull;
    key_T = pT >= 0 ? key_at<E>(key, pT) : ~0ull;
}

// Sweep 1: lower bound of each row's T-th score, into b1[32].
template <typename DT, int D, int TT>
__device__ void threshold_sweep(const Frag<DT, D> &fa, const DT *Kg, int n_k, int n_blk,
                                const int (&nrow)[16], int T, int hh, int l32, float *b1)
{
    float top[16][TT];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int j = 0; j < TT; ++j) top[i][j] = -INFINITY;
    for (int blk = 0; blk < n_blk; ++blk) {
        const int col = (blk << 5) + l32;
        Frag<DT, D> fb;
        if (col < n_k)
            fb.load(Kg + (int64_t)col * D, hh);
        else
            fb.zero();
        f32x16_t acc = {};
        acc = Frag<DT, D>::mma(fa, fb, acc);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            float x = (col < nrow[i]) ? acc[i] : -INFINITY;
#pragma unroll
            for (int j = 0; j < TT; ++j) {
                const float hi = fmaxf(top[i][j], x);
                x = fminf(top[i][j], x);
                top[i][j] = hi;
            }
        }
    }
    const int need = (T + TT - 1) / TT;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const float w = sort32_desc(top[i][TT - 1], l32);
        const float bound = __shfl(w, (hh << 5) + need - 1, 64);
        if (l32 == 0) b1[acc_row(i, hh)] = bound;
    }
}

// Sweep 2: append the scores that reach each row's (score, id) threshold to
// the row's LDS list in chunk-id order; cnt receives the number that did
// (entries beyond CAP are counted but not stored).
template <typename DT, int D, int CAP>
__device__ void collect_sweep(const Frag<DT, D> &fa, const DT *Kg, int n_k, int n_blk,
                              const int (&nrow)[16], int hh, int l32, const float *th_s,
                              const int32_t *th_id, float *bs, int32_t *bi, int32_t *cnt_s)
{
    float ths[16];
    int thi[16], cnt[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int r = acc_row(i, hh);
        ths[i] = th_s[r];
        thi[i] = th_id[r];
        cnt[i] = 0;
    }
    const uint32_t below = lanemask_lt32(l32);
    for (int blk = 0; blk < n_blk; ++blk) {
        const int col = (blk << 5) + l32;
        Frag<DT, D> fb;
        if (col < n_k)
            fb.load(Kg + (int64_t)col * D, hh);
        else
            fb.zero();
        f32x16_t acc = {};
        acc = Frag<DT, D>::mma(fa, fb, acc);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const float s = acc[i];
            const bool ok = (col < nrow[i]) && (s > ths[i] || (s == ths[i] && col <= thi[i]));
            const uint64_t mk = __ballot(ok);
            const uint32_t mh = hh ? (uint32_t)(mk >> 32) : (uint32_t)mk;
            const int slot = cnt[i] + __popc(mh & below);
            if (ok && slot < CAP) {
                const int r = acc_row(i, hh);
                bs[r * CAP + slot] = (s == 0.0f) ? 0.0f : s;
                bi[r * CAP + slot] = col;
            }
            cnt[i] += __popc(mh);
        }
    }
    if (l32 == 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i) cnt_s[acc_row(i, hh)] = cnt[i];
    }
}

template <typename DT, int D, int CAP, int TT>
__global__ __launch_bounds__(64) void route_kernel(RouteArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    float *bs = reinterpret_cast<float *>(smem);
    int32_t *bi = reinterpret_cast<int32_t *>(bs + kTileRows * CAP);
    uint32_t *bm = reinterpret_cast<uint32_t *>(bi + kTileRows * CAP);

    __shared__ int32_t row_i[kTileRows], row_n[kTileRows], row_g[kTileRows];
    __shared__ int32_t n_sel[kTileRows], cnt_s[kTileRows], th_id[kTileRows];
    __shared__ float th_s[kTileRows], b1_s[kTileRows];
    __shared__ int32_t s_head;

    const int lane = threadIdx.x, hh = lane >> 5, l32 = lane & 31;
    const int mode = a.mode;
    const int T = a.k + a.m;
    const int group = a.n_heads / a.n_kv_heads;
    const int nkw = (a.n_k + 31) >> 5;
    const int c_sent = a.m + a.r;
    const int ntiles = (mode == MODE_REROUTE) ? a.tile_base[a.n_heads] : a.n_heads * a.tiles_per_head;

    if (a.pairs_out && mode != MODE_REROUTE && blockIdx.x == 0 && lane == 0) *a.pairs_out = a.pairs_value;

    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        // ---------------------------------------------------- rows of the tile
        int h, t;
        if (mode == MODE_REROUTE) {
            if (lane == 0) s_head = 0;
            __syncthreads();
            for (int hb = lane; hb < a.n_heads; hb += 64)
                if (a.tile_base[hb] <= tile && tile < a.tile_base[hb + 1]) s_head = hb;
            __syncthreads();
            h = s_head;
            t = tile - a.tile_base[h];
        } else {
            h = tile / a.tiles_per_head;
            t = tile % a.tiles_per_head;
        }
        if (lane < kTileRows) {
            row_g[lane] = -1;
            row_i[lane] = 0;
            row_n[lane] = 0;
        }
        __syncthreads();
        if (mode == MODE_REROUTE) {
            const int lo = t * kTileRows, hi = lo + kTileRows;
            const uint8_t *fl = a.flags + (int64_t)h * a.n_q;
            int run = 0;
            for (int base = 0; base < a.n_q && run < hi; base += 64) {
                const int i = base + lane;
                const bool f = (i < a.n_q) && fl[i] != 0;
                const uint64_t mk = __ballot(f);
                const int rank = run + __popcll(mk & ((1ull << lane) - 1ull));
                if (f && rank >= lo && rank < hi) {
                    row_i[rank - lo] = i;
                    row_g[rank - lo] = h * a.n_q + i;
                    if (a.ids_out) a.ids_out[(int64_t)h * a.n_q + rank] = i;
                }
                run += __popcll(mk);
            }
        } else if (lane < kTileRows) {
            const int i = t * kTileRows + lane;
            if (i < a.n_q) {
                row_i[lane] = i;
                row_g[lane] = h * a.n_q + i;
            }
        }
        __syncthreads();
        if (lane < kTileRows && row_g[lane] >= 0) {
            const int i = row_i[lane];
            row_n[lane] = a.causal ? min(i + 1, a.n_k) : a.n_k;
        }
        __syncthreads();

        int ncols = lane < kTileRows ? row_n[lane] : 0;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) ncols = max(ncols, __shfl_xor(ncols, off, 64));
        const int n_blk = (ncols + 31) >> 5;

        int nrow[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) nrow[i] = row_n[acc_row(i, hh)];
        const DT *Kg = reinterpret_cast<const DT *>(a.K) + (int64_t)(h / group) * a.n_k * D;
        Frag<DT, D> fa;
        if (row_g[l32] >= 0)
            fa.load(reinterpret_cast<const DT *>(a.Q) + (int64_t)row_g[l32] * D, hh);
        else
            fa.zero();

        // ------------------------------------------------------ thresholds
        bool have_b1 = false;
        if (mode == MODE_REROUTE) {
            if (lane < kTileRows) {
                float th = -INFINITY;
                if (row_g[lane] >= 0) {
                    const float v = a.theta[row_g[lane]];
                    if (isfinite(v)) th = v - fabsf(v) * (1.0f / 4096.0f);
                }
                th_s[lane] = th;
                th_id[lane] = INT_MAX;
            }
        } else {
            threshold_sweep<DT, D, TT>(fa, Kg, a.n_k, n_blk, nrow, T, hh, l32, b1_s);
            have_b1 = true;
            __syncthreads();
            if (lane < kTileRows) {
                th_s[lane] = b1_s[lane];
                th_id[lane] = INT_MAX;
            }
        }
        __syncthreads();

        // ------------------------------------------------------ collection
        for (int it = 0;; ++it) {
            collect_sweep<DT, D, CAP>(fa, Kg, a.n_k, n_blk, nrow, hh, l32, th_s, th_id, bs, bi, cnt_s);
            __syncthreads();
            bool under = false, over = false;
            if (lane < kTileRows && row_g[lane] >= 0) {
                const int c = cnt_s[lane];
                under = c < min(T, row_n[lane]);
                over = c > CAP;
            }
            const uint64_t mu = __ballot(under), mo = __ballot(over);
            if ((mu | mo) == 0ull || it >= kMaxFixIters) break;
            if (mu) {
                if (!have_b1) {
                    threshold_sweep<DT, D, TT>(fa, Kg, a.n_k, n_blk, nrow, T, hh, l32, b1_s);
                    have_b1 = true;
                    __syncthreads();
                }
                if (under) {
                    th_s[lane] = b1_s[lane];
                    th_id[lane] = INT_MAX;
                }
            }
            uint64_t todo = mo;
            while (todo) {
                const int r = __ffsll((unsigned long long)todo) - 1;
                todo &= todo - 1ull;
                uint64_t kk_key, kT_key;
                select_bounds<CAP>(bs + r * CAP, bi + r * CAP, CAP, T, T, lane, kk_key, kT_key);
                if (lane == 0) {
                    th_s[r] = key_score(kT_key);
                    th_id[r] = key_id(kT_key);
                }
            }
            __syncthreads();
        }

        // ------------------------------------------------ selection, output
        for (int r = 0; r < kTileRows; ++r) {
            if (row_g[r] < 0) continue;
            const int64_t row = row_g[r];
            const int c = min(cnt_s[r], CAP);
            uint64_t key_k, key_T;
            select_bounds<CAP>(bs + r * CAP, bi + r * CAP, c, a.k, T, lane, key_k, key_T);
            if (mode != MODE_FULL) {
                for (int w = lane; w < nkw; w += 64) bm[r * nkw + w] = 0u;
                __syncthreads();
            }
            int nR = 0, nN = 0;
            for (int base = 0; base < c; base += 64) {
                const int idx = base + lane;
                const bool v = idx < c;
                const float s = v ? bs[r * CAP + idx] : 0.0f;
                const int id = v ? bi[r * CAP + idx] : 0;
                const uint64_t key = v ? rank_key(s, id) : 0ull;
                const bool inR = v && key >= key_k;
                const bool inN = v && !inR && key >= key_T;
                const uint64_t mR = __ballot(inR), mN = __ballot(inN);
                const uint64_t below = (1ull << lane) - 1ull;
                if (inR) {
                    const int pos = nR + __popcll(mR & below);
                    if (a.led_routes) a.led_routes[row * a.k + pos] = id;
                    if (a.routes_out) a.routes_out[row * a.k + pos] = id;
                    if (a.scores_out) a.scores_out[row * a.k + pos] = s;
                }
                if (inN) {
                    const int pos = nN + __popcll(mN & below);
                    a.led_sent[row * c_sent + pos] = id;
                }
                if (mode != MODE_FULL && (inR || inN)) atomicOr(&bm[r * nkw + (id >> 5)], 1u << (id & 31));
                nR += __popcll(mR);
                nN += __popcll(mN);
            }
            for (int j = nR + lane; j < a.k; j += 64) {
                if (a.led_routes) a.led_routes[row * a.k + j] = -1;
                if (a.routes_out) a.routes_out[row * a.k + j] = -1;
                if (a.scores_out) a.scores_out[row * a.k + j] = -INFINITY;
            }
            if (mode != MODE_FULL)
                for (int j = nN + lane; j < a.m; j += 64) a.led_sent[row * c_sent + j] = -1;
            if (lane == 0) n_sel[r] = nR + nN;
        }
        __syncthreads();

        // ------------------------------------------------ random sentinels
        if (mode != MODE_FULL && lane < kTileRows && row_g[lane] >= 0) {
            const int r = lane;
            const int64_t row = row_g[r];
            const int ni = row_n[r];
            const int pool = ni - n_sel[r];
            int32_t *out = a.led_sent + row * c_sent + a.m;
            uint32_t *bmr = bm + r * nkw;
            if (pool <= a.r) {
                int w = 0;
                for (int wd = 0; wd * 32 < ni; ++wd) {
                    uint32_t z = ~bmr[wd];
                    const int lim = ni - wd * 32;
                    if (lim < 32) z &= (1u << lim) - 1u;
                    while (z) {
                        out[w++] = wd * 32 + __ffs(z) - 1;
                        z &= z - 1u;
                    }
                }
                for (; w < a.r; ++w) out[w] = -1;
            } else {
                const uint64_t h0 = sm64(sm64(sm64(a.seed) ^ (uint64_t)(uint32_t)a.layer) ^ (uint64_t)row);
                for (int s = 0; s < a.r; ++s) {
                    const uint64_t hs = sm64(h0 ^ (uint64_t)s);
                    int chosen = -1;
                    for (int at = 0; at < 64; ++at) {
                        const int x = (int)(sm64(hs ^ (uint64_t)at) % (uint64_t)ni);
                        if (!((bmr[x >> 5] >> (x & 31)) & 1u)) {
                            chosen = x;
                            break;
                        }
                    }
                    if (chosen < 0) {
                        int y = (int)(sm64(hs ^ 64ull) % (uint64_t)(pool - s));
                        for (int wd = 0; chosen < 0 && wd < nkw; ++wd) {
                            const int lim = ni - wd * 32;
                            if (lim <= 0) break;
                            uint32_t z = ~bmr[wd];
                            if (lim < 32) z &= (1u << lim) - 1u;
                            const int pc = __popc(z);
                            if (y < pc) {
                                for (int q = 0; q < y; ++q) z &= z - 1u;
                                chosen = wd * 32 + __ffs(z) - 1;
                            } else {
                                y -= pc;
                            }
                        }
                    }
                    if (chosen >= 0) bmr[chosen >> 5] |= 1u << (chosen & 31);
                    out[s] = chosen;
                }
            }
            a.led_build[row] = a.layer;
            a.led_age[row] = 0;
        }
        __syncthreads();
    }
}

template <typename DT, int D, int CAP, int TT>
hipError_t launch_t(const RouteArgs &a, int grid, hipStream_t stream)
{
    const size_t lds = (size_t)kTileRows * CAP * 8 + (size_t)kTileRows * ((a.n_k + 31) / 32) * 4;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&route_kernel<DT, D, CAP, TT>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((route_kernel<DT, D, CAP, TT>), dim3(grid), dim3(64), lds, stream, a);
    return hipGetLastError();
}

template <typename DT, int D>
hipError_t launch_d(const RouteArgs &a, int grid, hipStream_t stream)
{
    if (a.k + a.m > 64) return launch_t<DT, D, 256, 4>(a, grid, stream);
    return launch_t<DT, D, 128, 2>(a, grid, stream);
}

}  // namespace

bool route_supported(int dtype, int d, int T)
{
    if (T < 1 || T > 128) return false;
    if (dtype == 0) return d == 32 || d == 64 || d == 128;
    if (dtype == 1) return d == 32 || d == 64 || d == 128 || d == 256;
    return false;
}

hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream)
{
    if (dtype == 0) {
        switch (a.d) {
        case 32: return launch_d<float, 32>(a, grid, stream);
        case 64: return launch_d<float, 64>(a, grid, stream);
        case 128: return launch_d<float, 128>(a, grid, stream);
        default: break;
        }
    } else {
        switch (a.d) {
        case 32: return launch_d<bf16_t, 32>(a, grid, stream);
        case 64: return launch_d<bf16_t, 64>(a, grid, stream);
        case 128: return launch_d<bf16_t, 128>(a, grid, stream);
        case 256: return launch_d<bf16_t, 256>(a, grid, stream);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
