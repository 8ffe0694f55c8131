// Row-wise GEMM + TopK routing for gfx950 (RouteRelay, arXiv 2609.07306).
//
// One kernel serves four callers:
//   MODE_FULL    -- full routing of every row, Eq. (1)-(2) (the baseline);
//   MODE_ANCHOR  -- full routing plus the ledger build of Sec. 3.1: the
//                   chunks ranked k+1..k+m become near-miss sentinels and r
//                   random sentinels are drawn from what is left;
//   MODE_REROUTE -- the same for the rows a relay layer flagged (Sec. 3.2,
//                   row-selective refresh of Sec. 4.2), read per head from
//                   the flag array in ascending row order;
//   MODE_RELAY   -- the one-pass relay: the threshold sweep also rescores
//                   each row's ledger (Eq. (5)-(7)) from per-row bitmaps,
//                   the trigger of Eq. (8) flags the row, and the tile's
//                   flagged rows are routed as in MODE_REROUTE.
//
// A workgroup owns a tile of 32*NW query rows of one head and runs KS waves
// per 32-row block: the KS waves of a block split the key range between them
// (the 128-row tiles run 8 waves, two per SIMD, so one wave's memory and LDS
// latency hides under the other's work).  The padded key range is cut into
// 2*KS segments of equal length; at stage st, wave split p multiplies the
// 32-key tile made of keys st*16 .. st*16+15 of segments 2p and 2p+1.  The
// tiles of all splits of a stage go global -> registers two stages ahead and
// registers -> LDS one stage ahead (double-buffered, rows padded and swizzled
// so both halves of a wave read distinct bank groups), and the MFMAs of
// stage st+1 are issued before the epilogue of stage st.  The score matrix is
// never stored.
//
// Every product is the transposed one (A = keys, B = queries, the 32x32x16
// bf16 or 32x32x2 f32 MFMA), so lane (r, hh) of wave split p holds row r of
// the block and 16 consecutive keys of segment 2p+hh per stage.  Selecting
// the T = k + m best chunks of each row takes two sweeps over the keys:
//   1. threshold: each lane keeps, per register slot, the top TT scores of
//      the keys that pass through the slot (TT = 2: one max and one med3 per
//      score).  The union U of a row's 2*KS*16*TT kept scores holds at least
//      T of the row's scores, so any v with |{u in U: u >= v}| >= T is at
//      most the row's T-th score; the lists are regrouped through LDS so that
//      a few neighbouring lanes of one wave hold a row's U, and v is raised
//      by bisection from U's smallest finite entry toward the row maximum.
//   2. collection: every lane appends the scores of its segment that reach
//      its row's threshold, with their ids, to the segment's sub-list of the
//      row; a row's sub-lists in segment order are its candidates in id
//      order.  A sub-list that overflows its share of the row region is
//      repaired: if the row's candidates fit the whole region, the sweep is
//      repeated with the sub-lists placed at the exclusive prefix of their
//      counts; otherwise the threshold is raised by bisection in the
//      order-preserving integer image of the scores, and when the T-th score
//      is pinned (bisection bounds adjacent) the id cut of its ties is found
//      by a second bisection, so that exactly T chunks are admitted.  Repairs
//      change work, never results.
// Selection runs on four lanes per row (lanes l, l+16, l+32, l+48 of a
// wave, every wave of the workgroup): a bitonic network over the first NET
// candidates, sorted in quarters and merged across the row's lanes, plus
// insertion of any further ones, gives the k-th and T-th scores; each lane
// then assigns R and the near-miss set over a quarter of the id-ordered
// candidates (equal scores rank the lower id first), writing both sorted by
// id at offsets from the counts of the quarters before it.  The random
// sentinels are drawn by the same four lanes: a pool of at most half the
// valid chunks by rank (the y-th free chunk of a per-row bitmap of R, N and
// earlier draws), a larger one by counter-hash probes reduced modulo n_i
// (Barrett), rejected with the bitmap (exact up to 4096 chunks where the
// row's candidate region holds 128 words, else 2048; beyond that a filter
// on the id modulo the bitmap's width whose hits are checked by binary
// search of R and N and a scan of the earlier draws).  Slots whose outcome
// depends only on their own hash (first probes, rank draws' ranks) are
// hashed four at a time and decided in slot order, so the draws are those of
// one lane deciding the slots one by one.
//
// This header holds the kernel template; each rr_route_<type>_<mode>.hip
// translation unit instantiates one input type and caller, so the library
// builds in parallel and each caller is a kernel of its own in a trace.
#pragma once

#include <limits.h>
#include <type_traits>
#include <math.h>

#include "rr_device.hpp"
#include "rr_internal.hpp"

namespace rr {
namespace route_detail {

constexpr int kMaxFixIters = 64;  // default cap on collection sweeps per tile (score + id bisection need <= 50)
constexpr int kBisect = 10;       // bisection steps of the threshold bound
constexpr uint32_t kSeedSlack = 8;  // orders by which a reroute widens the rescoring pass's bound and maximum
constexpr int kPrefetch = 2;      // key stages in flight ahead of the MFMA

// row states of the collection loop
constexpr int kSweep = 0;   // a score threshold is applied
constexpr int kTieCut = 1;  // the T-th score is pinned; bisecting the id cut of its ties
constexpr int kDone = 2;    // candidates complete in LDS

// Descending bitonic sorting network on a register array (one row per lane),
// generated by template recursion so every element index is a constant and
// the array stays in registers.
template <int N, int KK, int J, int I>
struct BitonicPairs {
    __device__ static __forceinline__ void run(float (&v)[N])
    {
        constexpr int L = I ^ J;
        if constexpr (L > I) {
            const float x = v[I], y = v[L];
            if constexpr ((I & KK) == 0) {
                v[I] = fmaxf(x, y);
                v[L] = fminf(x, y);
            } else {
                v[I] = fminf(x, y);
                v[L] = fmaxf(x, y);
            }
        }
        if constexpr (I + 1 < N) BitonicPairs<N, KK, J, I + 1>::run(v);
    }
};

template <int N, int KK, int J>
struct BitonicStages {
    __device__ static __forceinline__ void run(float (&v)[N])
    {
        BitonicPairs<N, KK, J, 0>::run(v);
        if constexpr (J > 1) BitonicStages<N, KK, J / 2>::run(v);
    }
};

template <int N, int KK>
struct BitonicMerges {
    __device__ static __forceinline__ void run(float (&v)[N])
    {
        BitonicStages<N, KK, KK / 2>::run(v);
        if constexpr (KK < N) BitonicMerges<N, KK * 2>::run(v);
    }
};

template <int N>
__device__ __forceinline__ void sort_desc(float (&v)[N])
{
    BitonicMerges<N, 2>::run(v);
}

// Descending bitonic merge of a bitonic register array.
template <int N>
__device__ __forceinline__ void merge_desc(float (&v)[N])
{
    BitonicStages<N, N, N / 2>::run(v);
}

// v[idx] of a descending array, as the minimum of its first idx+1 entries (a
// compare-select chain on the index would be lowered to a stack array).
template <int N>
__device__ __forceinline__ float sorted_at(const float (&v)[N], int idx)
{
    float x = v[0];
#pragma unroll
    for (int i = 1; i < N; ++i) x = fminf(x, (i <= idx) ? v[i] : INFINITY);
    return x;
}

template <int N>
__device__ __forceinline__ int count_gt(const float (&v)[N], float x)
{
    int c = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) c += (v[i] > x) ? 1 : 0;
    return c;
}

template <int N>
__device__ __forceinline__ int count_eq(const float (&v)[N], float x)
{
    int c = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) c += (v[i] == x) ? 1 : 0;
    return c;
}

// Keep the TT largest of top[0..TT) u {x}; top is sorted descending.
template <int TT>
__device__ __forceinline__ void top_insert(float (&top)[TT], float x)
{
    float prev = top[0];
    top[0] = fmaxf(prev, x);
#pragma unroll
    for (int j = 1; j < TT; ++j) {
        const float cur = top[j];
        top[j] = __builtin_amdgcn_fmed3f(prev, cur, x);
        prev = cur;
    }
}

template <typename DT, int D, int NW, int KS, int TT, int NETW, int CAPQ>
struct RT {
    using DType = DT;
    static constexpr int DIM = D, NW_ = NW, KS_ = KS, TT_ = TT, CAPQ_ = CAPQ;
    static constexpr int NWV = NW * KS;            // waves
    static constexpr int NT = 64 * NWV;            // threads
    static constexpr int BM = 32 * NW;             // rows per tile
    static constexpr int NSEG = 2 * KS;            // key segments = sub-lists per row
    static constexpr int ROWB = D * (int)sizeof(DT);
    static constexpr int BSTR = ROWB + 16;         // padded LDS key-row stride (odd count of 16 B)
    static_assert((BSTR / 16) % 2 == 1, "row stride must be an odd number of 16-byte bank groups");
    static constexpr int BT = 32 * BSTR;           // one 32-key tile
    static constexpr int ST = KS * BT;             // one stage: a tile per key split
    static constexpr int TCH = 32 * ROWB / 16;     // 16-byte pieces of a tile
    static constexpr int CHUNKS = KS * TCH;        // ... of a stage
    static constexpr int PER_T = (CHUNKS + NT - 1) / NT;
    static constexpr int NET = NETW;               // candidates sorted by the network
    static constexpr int CAPR = NSEG * CAPQ;       // candidate capacity of a row
    static_assert(CAPR >= NET, "a row region holds at least the network's candidates");
    static constexpr int SS = CAPR + 1;            // candidate row stride (floats, odd); slot CAPR is a dummy
    static constexpr int SI = CAPR + 2;            // candidate row stride (u16 ids)
    static constexpr int NU = NSEG * 16 * TT;      // kept scores per row after the threshold sweep
    static constexpr int LPR = NT / BM;            // lanes per row in the bound step
    static constexpr int UPL = NU / LPR;           // kept scores per bound lane
    static constexpr int UST = NU + 4;             // LDS row stride of the kept scores (16-byte rows)
    // words of a row's membership bitmap in its candidate region (SS floats,
    // odd, so rows fall in different banks): exact for n_i <= 32 * BMW
    static constexpr int BMW = (SS - 1 >= 128) ? 128 : 64;
    static_assert(BMW < SS, "a row's bitmap fits its candidate region");
    static_assert(NU % (4 * LPR) == 0 && (LPR & (LPR - 1)) == 0, "bound lanes take whole float4 groups");
};

// LDS slot of key-tile row t.  Rows 16..31 are XOR-swizzled by 12 so that
// each group of 8 (or 16) consecutive lanes reads rows in distinct bank
// groups in the transposed product (lanes read rows 0-3, 16-19, 4-7, 20-23,
// ...); the padded row stride is an odd number of 16-byte bank groups.
__device__ __forceinline__ int tile_slot(int t) { return t ^ ((t >> 4) * 12); }

// Tile row read by lane l32 for the transposed (A = keys) product: output
// register i of half hh then holds tile row 16*hh + i.
__device__ __forceinline__ int transposed_row(int l32)
{
    return (l32 & 4) ? 16 + 4 * (l32 >> 3) + (l32 & 3) : 4 * (l32 >> 3) + (l32 & 3);
}

// Key held by row tr (0..31) of split p's tile at stage st: rows 0..15 are
// keys st*16 .. st*16+15 of segment 2p, rows 16..31 the same of segment 2p+1.
__device__ __forceinline__ int stage_key(int st, int p, int tr, int seg)
{
    return (2 * p + (tr >> 4)) * seg + 16 * st + (tr & 15);
}

// Global -> registers: this thread's pieces of key stage st.  Every load is
// issued: the stage, the piece and the key are clamped to valid values (keys
// past n_k and stages past the last read real rows whose scores every
// epilogue masks or skips), so the loads carry no branches and the compiler
// can wait for exactly the oldest.
template <class C>
__device__ __forceinline__ void key_gload(u32x4_t (&breg)[C::PER_T], const unsigned char *Kg, int n_k, int seg, int st,
                                          int tid)
{
#pragma unroll
    for (int u = 0; u < C::PER_T; ++u) {
        int ch = tid + u * C::NT;
        if constexpr (C::CHUNKS % C::NT != 0) ch = min(ch, C::CHUNKS - 1);
        const int p = ch / C::TCH, rem = ch - p * C::TCH;
        const int tr = rem / (C::ROWB / 16), off = rem - tr * (C::ROWB / 16);
        const int key = min(stage_key(st, p, tr, seg), n_k - 1);
        breg[u] = *reinterpret_cast<const u32x4_t *>(Kg + (int64_t)key * C::ROWB + off * 16);
    }
}

// Registers -> LDS stage slot buf (threads past the last piece repeat it with
// identical data).
template <class C>
__device__ __forceinline__ void key_lstore(const u32x4_t (&breg)[C::PER_T], unsigned char *bt, int buf, int tid)
{
#pragma unroll
    for (int u = 0; u < C::PER_T; ++u) {
        int ch = tid + u * C::NT;
        if constexpr (C::CHUNKS % C::NT != 0) ch = min(ch, C::CHUNKS - 1);
        const int p = ch / C::TCH, rem = ch - p * C::TCH;
        const int tr = rem / (C::ROWB / 16), off = rem - tr * (C::ROWB / 16);
        *reinterpret_cast<u32x4_t *>(bt + buf * C::ST + p * C::BT + tile_slot(tr) * C::BSTR + off * 16) = breg[u];
    }
}

// Calls f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>).
template <int I, int N>
struct StaticFor {
    template <class F>
    __device__ static __forceinline__ void run(F &&f)
    {
        if constexpr (I < N) {
            f(std::integral_constant<int, I>{});
            StaticFor<I + 1, N>::run(f);
        }
    }
};

template <int N, class F>
__device__ __forceinline__ void static_for(F &&f)
{
    StaticFor<0, N>::run(f);
}

// acc = K_tile x Q_rows: lane (r, hh) gets row r and the 16 keys of its
// segment; the plain d-ordered product.
template <typename DT, int D>
__device__ __forceinline__ f32x16_t tile_product(const Frag<DT, D> &fq, const Frag<DT, D> &fk)
{
    f32x16_t out = f32x16_t{};
#pragma unroll
    for (int s = 0; s < Frag<DT, D>::NS; ++s) out = Frag<DT, D>::mma_step(fk, fq, out, s);
    return out;
}

// Scheduling hint: alternate the NM MFMAs of the next stage with groups of K
// epilogue instructions (VALU or LDS writes) of the current one, so the MFMA
// chain runs under the epilogue.
template <int NM, int K>
__device__ __forceinline__ void interleave_mfma()
{
#pragma unroll
    for (int j = 0; j < NM; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002 | 0x200, K, 0);
    }
}

// One pass over the key stages 0..nb-1.  epi.step(st, acc, next, fq, fk,
// full) runs the epilogue of stage st on acc while issuing the MFMAs of
// stage st+1 (fragments fk) into next; full = every key of this wave's tile
// of stage st is valid for every row of the wave.
//
// Per stage st: st+1's MFMAs run under st's epilogue, st+2 moves registers ->
// LDS into the slot st used, st+2+PF is requested from global memory, and
// after the barrier the fragments of st+2 are read.  A slot is rewritten only
// after the barrier that follows the MFMAs reading it.  The two accumulator
// sets alternate, so no copies are needed.  Past the last stage the loads
// repeat the last stage and the extra products are never used: the
// steady-state loop has no conditional memory operations.
template <typename DT, int D, class C, class Epi>
__device__ __forceinline__ void sweep_keys(const Frag<DT, D> &fq, const unsigned char *Kg, int n_k, int seg, int nb,
                                           int full_stages, int tid, int p, int hh, int l32, unsigned char *bt,
                                           Epi &epi)
{
    constexpr int PF = kPrefetch;
    static_assert(PF % 2 == 0, "accumulator sets alternate through the unrolled loop");
    const int last = nb - 1;
    const unsigned char *lp = bt + p * C::BT + tile_slot(transposed_row(l32)) * C::BSTR;
    u32x4_t breg[PF][C::PER_T];
#pragma unroll
    for (int u = 0; u < PF; ++u) key_gload<C>(breg[u], Kg, n_k, seg, min(u, last), tid);
    key_lstore<C>(breg[0], bt, 0, tid);
    key_gload<C>(breg[0], Kg, n_k, seg, min(PF, last), tid);
    key_lstore<C>(breg[1], bt, 1, tid);
    key_gload<C>(breg[1], Kg, n_k, seg, min(PF + 1, last), tid);
    __syncthreads();
    Frag<DT, D> fk;
    fk.load(reinterpret_cast<const DT *>(lp), hh);
    f32x16_t acc[2];
    acc[0] = tile_product(fq, fk);
    acc[1] = acc[0];
    fk.load(reinterpret_cast<const DT *>(lp + C::ST), hh);
    __syncthreads();  // stages 0 and 1 are read by every wave before slot 0 is rewritten
    // U = st mod PF is a compile-time constant, so the register ring is
    // indexed statically
    auto block = [&](int st, auto uc) __attribute__((always_inline)) {
        constexpr int U = decltype(uc)::value;
        epi.step(st, acc[U & 1], acc[(U + 1) & 1], fq, fk, st < full_stages);
        key_lstore<C>(breg[(U + 2) % PF], bt, st & 1, tid);
        key_gload<C>(breg[(U + 2) % PF], Kg, n_k, seg, min(st + 2 + PF, last), tid);
        __syncthreads();
        fk.load(reinterpret_cast<const DT *>(lp + (st & 1) * C::ST), hh);
    };
    int s0 = 0;
    for (; s0 + PF <= nb; s0 += PF) {
        static_for<PF>([&](auto uc) __attribute__((always_inline)) { block(s0 + decltype(uc)::value, uc); });
    }
    static_for<PF - 1>([&](auto uc) __attribute__((always_inline)) {
        if (s0 + decltype(uc)::value < nb) block(s0 + decltype(uc)::value, uc);
    });
}

// The same pass with the key fragments double-buffered in registers, for
// kernels with the registers to spare: the LDS reads of stage st+2 are
// issued at the top of block st and complete under the MFMAs of stage st+1
// and the epilogue of stage st, instead of between the barrier and the next
// MFMA.  Block st reads stage st+2 from slot st&1 (stored in block st-1) and
// stores stage st+3 into slot (st+1)&1, whose stage st+1 every wave read
// before the previous barrier (a workgroup barrier waits for the wave's LDS
// reads).  The prologue keeps stages 0 and 1 in registers and stage 2 in slot
// 0; stages past the last are clamped reloads whose products are never used.
// The caller issues the loads of stages 0 and 1 into breg (sweep_db_first),
// so that they can be in flight during its own set-up.
template <class C>
__device__ __forceinline__ void sweep_db_first(u32x4_t (&breg)[2][C::PER_T], const unsigned char *Kg, int n_k,
                                               int seg, int nb, int tid)
{
    key_gload<C>(breg[0], Kg, n_k, seg, 0, tid);
    key_gload<C>(breg[1], Kg, n_k, seg, min(1, nb - 1), tid);
}

template <typename DT, int D, class C, class Epi>
__device__ __forceinline__ void sweep_keys_db(const Frag<DT, D> &fq, const unsigned char *Kg, int n_k, int seg, int nb,
                                              int full_stages, int tid, int p, int hh, int l32, unsigned char *bt,
                                              u32x4_t (&breg)[2][C::PER_T], Epi &epi)
{
    constexpr int PF = kPrefetch;
    static_assert(PF == 2, "the register ring and the two LDS slots advance in step");
    const int last = nb - 1;
    const unsigned char *lp = bt + p * C::BT + tile_slot(transposed_row(l32)) * C::BSTR;
    key_lstore<C>(breg[0], bt, 0, tid);
    key_lstore<C>(breg[1], bt, 1, tid);
    key_gload<C>(breg[0], Kg, n_k, seg, min(2, last), tid);
    key_gload<C>(breg[1], Kg, n_k, seg, min(3, last), tid);
    __syncthreads();
    Frag<DT, D> fk[2];
    fk[0].load(reinterpret_cast<const DT *>(lp), hh);
    fk[1].load(reinterpret_cast<const DT *>(lp + C::ST), hh);
    f32x16_t acc[2];
    acc[0] = tile_product(fq, fk[0]);
    acc[1] = acc[0];
    __syncthreads();  // stages 0 and 1 are in every wave's registers
    key_lstore<C>(breg[0], bt, 0, tid);
    key_gload<C>(breg[0], Kg, n_k, seg, min(4, last), tid);
    __syncthreads();  // stage 2 is in slot 0
    auto block = [&](int st, auto uc) __attribute__((always_inline)) {
        constexpr int U = decltype(uc)::value;  // st & 1
        fk[U].load(reinterpret_cast<const DT *>(lp + U * C::ST), hh);
        epi.step(st, acc[U], acc[U ^ 1], fq, fk[U ^ 1], st < full_stages);
        key_lstore<C>(breg[U ^ 1], bt, U ^ 1, tid);
        key_gload<C>(breg[U ^ 1], Kg, n_k, seg, min(st + 5, last), tid);
        __syncthreads();
    };
    int s0 = 0;
    for (; s0 + 2 <= nb; s0 += 2) {
        static_for<2>([&](auto uc) __attribute__((always_inline)) { block(s0 + decltype(uc)::value, uc); });
    }
    if (s0 < nb) block(s0, std::integral_constant<int, 0>{});
}

// Threshold-sweep epilogue: per register slot, the top TT scores of the keys
// of this lane's segment that pass through the slot (invalid keys count as
// -inf).
template <int TT>
struct TopEpi {
    float top[16][TT];
    int nrow;   // valid keys of the lane's row (0: padding row)
    int sbase;  // first key of the lane's segment

    template <class F>
    __device__ __forceinline__ void step(int st, const f32x16_t &acc, f32x16_t &next, const F &fq, const F &fk,
                                         bool full)
    {
        next = tile_product(fq, fk);
        if (full) {
#pragma unroll
            for (int i = 0; i < 16; ++i) top_insert<TT>(top[i], acc[i]);
            interleave_mfma<F::NS, (16 * TT + F::NS - 1) / F::NS>();
        } else {
            const int vlim = nrow - (sbase + 16 * st);  // keys sbase + 16 st + i are valid for i < vlim
#pragma unroll
            for (int i = 0; i < 16; ++i) top_insert<TT>(top[i], (i < vlim) ? acc[i] : -INFINITY);
        }
    }
};

// Relay threshold-sweep epilogue: TopEpi's kept scores, and the rescoring
// of the ledger's candidates on the same scores (Sec. 3.2 Eq. (6)-(7)):
// amin = min over the routed set R, bmax = max over the sentinel set C, from
// the row's ledger bitmaps ((R word, C word) per 32 keys): a score outside
// the set becomes +inf for the minimum, -inf for the maximum.
template <int TT>
struct RelayEpi {
    float top[16][TT];
    int nrow;   // valid keys of the lane's row (0: padding row)
    int sbase;  // first key of the lane's segment
    float amin, bmax;
    const uint2 *bmr;  // this lane's row bitmap
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
        next = tile_product(fq, fk);
        const uint32_t sh = (uint32_t)(k0 & 16);
        const uint32_t mr = wv.x >> sh, mc = wv.y >> sh;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const uint32_t xb = __float_as_uint(acc[i]);
            const uint32_t nr = (uint32_t)((int32_t)(mr << (31 - i)) >> 31);  // all-ones where in R
            const uint32_t nc = (uint32_t)((int32_t)(mc << (31 - i)) >> 31);  // all-ones where in C
            amin = fminf(amin, __uint_as_float((xb & nr) | (0x7F800000u & ~nr)));
            bmax = fmaxf(bmax, __uint_as_float((xb & nc) | (0xFF800000u & ~nc)));
        }
        if (full) {
#pragma unroll
            for (int i = 0; i < 16; ++i) top_insert<TT>(top[i], acc[i]);
        } else {
            const int vlim = nrow - k0;  // keys k0 + i are valid for i < vlim
#pragma unroll
            for (int i = 0; i < 16; ++i) top_insert<TT>(top[i], (i < vlim) ? acc[i] : -INFINITY);
        }
        interleave_mfma<F::NS, (16 * (TT + 6) + F::NS - 1) / F::NS>();
    }
};

// The lane's 16 x TT kept scores -> its segment's part of the row's kept
// set in LDS (rows of UST floats).
template <class C, int TT>
__device__ __forceinline__ void store_kept(float *us, int myrow, int myseg, const float (&top)[16][TT])
{
    float *U = us + myrow * C::UST + myseg * 16 * TT;
#pragma unroll
    for (int q = 0; q < 4 * TT; ++q) {
        float4 x;
        x.x = top[(4 * q + 0) / TT][(4 * q + 0) % TT];
        x.y = top[(4 * q + 1) / TT][(4 * q + 1) % TT];
        x.z = top[(4 * q + 2) / TT][(4 * q + 2) % TT];
        x.w = top[(4 * q + 3) / TT][(4 * q + 3) % TT];
        reinterpret_cast<float4 *>(U)[q] = x;
    }
}

// Bound of the row's T-th score from its kept set U, LPR neighbouring
// threads per row (UPL kept scores each): any v with |{u in U : u >= v}| >= T
// is at most the row's T-th score; start from the smallest finite entry of U
// when U holds at least T of them (else -inf, which admits every valid chunk)
// and bisect toward the row maximum, which is U's largest entry.  Thread
// part 0 of row r stores the bound and the maximum into b1[r] and rmax[r].
template <class C>
__device__ __forceinline__ void bound_of_kept(const float *us, int tid, int T, float *b1, float *rmx)
{
    const int r = tid / C::LPR, part = tid % C::LPR;
    float u[C::UPL];
    const float4 *ur = reinterpret_cast<const float4 *>(us + r * C::UST + part * C::UPL);
#pragma unroll
    for (int q = 0; q < C::UPL / 4; ++q) {
        const float4 x = ur[q];
        u[4 * q] = x.x;
        u[4 * q + 1] = x.y;
        u[4 * q + 2] = x.z;
        u[4 * q + 3] = x.w;
    }
    float rmax = -INFINITY, umin = INFINITY;
    int nfin = 0;
#pragma unroll
    for (int q = 0; q < C::UPL; ++q) {
        const bool fin = u[q] > -INFINITY;
        rmax = fmaxf(rmax, u[q]);
        umin = fminf(umin, fin ? u[q] : INFINITY);
        nfin += fin ? 1 : 0;
    }
    // a row's four lanes are a DPP quad
    static_assert(C::LPR == 4 && C::NT % 64 == 0, "four bound lanes per row, whole waves");
    rmax = fmaxf(rmax, quad_xor1(rmax));
    umin = fminf(umin, quad_xor1(umin));
    nfin += quad_xor1(nfin);
    rmax = fmaxf(rmax, quad_xor2(rmax));
    umin = fminf(umin, quad_xor2(umin));
    nfin += quad_xor2(nfin);
    float lo = (nfin >= T) ? umin : -INFINITY, hi = rmax;
    if (lo > -INFINITY) {
        for (int it = 0; it < kBisect; ++it) {
            const float mid = lo + 0.5f * (hi - lo);
            // entries below mid, by the sign of u - mid: exact, u == mid gives
            // +0, and a difference too small to represent keeps its sign
            // (the count needs no compare results, whose reads stall)
            int neg = 0;
#pragma unroll
            for (int q = 0; q < C::UPL; ++q) neg += (int)(__float_as_uint(u[q] - mid) >> 31);
            int cnt = C::UPL - neg;
            cnt += quad_xor1(cnt);
            cnt += quad_xor2(cnt);
            if (cnt >= T)
                lo = mid;
            else
                hi = mid;
        }
    }
    if (part == 0) {
        b1[r] = lo;
        rmx[r] = rmax;
    }
}

// Collection-sweep epilogue: the lane appends the scores of its segment that
// reach its row's threshold to its sub-list.  A chunk is admitted when
// s > th, or s == th and its id is at most th_id; th_id is INT_MAX except
// in a tie cut, so the wave normally takes the one-compare path.  Appends
// past the sub-list's capacity run on into the row's later sub-lists, never
// past the row's dummy slot: a row with a sub-list over capacity is swept
// again with new placements, which rewrite all of its sub-lists, so the
// overrun entries are never read (and the other rows are untouched).
struct CollectEpi {
    float th;      // row threshold score (+inf: nothing is admitted)
    int th_id;     // row threshold id (INT_MAX: plain score threshold)
    int nrow;      // valid keys of the row (0: padding row)
    int sbase;     // first key of the lane's segment
    int cnt;       // entries admitted (may exceed the sub-list's capacity: overflow)
    int dum;       // the row's dummy slot, relative to ls / li
    float *ls;     // this lane's score sub-list
    uint16_t *li;  // this lane's id sub-list

    __device__ __forceinline__ void put(bool ok, float s, int key)
    {
        const int p = ok ? min(cnt, dum) : dum;
        ls[p] = s;
        li[p] = (uint16_t)key;
        cnt += ok ? 1 : 0;
    }

    // put(s >= th, s, key) with the test taken from the sign of s - th
    // (exact; a -inf threshold admits every score, +inf none): integer
    // arithmetic on the sign mask, no compare results to wait for
    __device__ __forceinline__ void put_ge(float s, int key)
    {
        const uint32_t below = (uint32_t)((int32_t)__float_as_uint(s - th) >> 31);  // all ones when s < th
        const int p = (int)min((uint32_t)cnt | below, (uint32_t)dum);
        ls[p] = s;
        li[p] = (uint16_t)key;
        cnt += 1 + (int)below;
    }

    template <class F>
    __device__ __forceinline__ void step(int st, const f32x16_t &acc, f32x16_t &next, const F &fq, const F &fk,
                                         bool full)
    {
        const int k0 = sbase + 16 * st;  // this lane's keys: k0 .. k0 + 15
        next = tile_product(fq, fk);
        if (full && __ballot(th_id - k0 < 15) == 0ull) {
#pragma unroll
            for (int i = 0; i < 16; ++i) put_ge(acc[i], k0 + i);
            interleave_mfma<F::NS, (16 * 7 + F::NS - 1) / F::NS>();
        } else {
            const int lim = th_id - k0;  // keys k0 + i with i <= lim admit s == th
            const int vlim = nrow - k0;  // keys k0 + i are valid for i < vlim
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                // (bitwise forms: the conditions compile to selects, not to
                // per-element branches)
                const float s = acc[i];
                put(((s > th) | ((s == th) & (i <= lim))) & (i < vlim), s, k0 + i);
            }
        }
    }
};

template <int MODE, typename DT, int D, int NW, int KS, int TT, int NETW, int CAPQ>
__global__ __launch_bounds__(64 * NW * KS) void route_kernel(RouteArgs a)
{
    using C = RT<DT, D, NW, KS, TT, NETW, CAPQ>;
    constexpr int BM = C::BM;
    constexpr int NET = C::NET;
    constexpr int NSEG = C::NSEG;
    constexpr int CAPR = C::CAPR;
    constexpr int STG = NET + 1;  // staging row stride (odd), holds k + m <= NET ids
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *bt = smem;  // [2][KS][32][BSTR] key tiles; later R / N staging
    float *ss = reinterpret_cast<float *>(smem + a.lds_region0);  // candidates; later the per-row bitmaps
    uint16_t *si = reinterpret_cast<uint16_t *>(ss + BM * C::SS);
    float *us = reinterpret_cast<float *>(smem);  // kept scores of the threshold sweep [BM][UST]

    __shared__ int32_t row_i[BM], row_n[BM], row_k[BM], row_g[BM], th_id[BM], cnt_hi[BM], rstate[BM], id_lo[BM], id_hi[BM];
    __shared__ float th_s[BM], b1_s[BM], rmax_s[BM];
    __shared__ uint32_t lo_k[BM], hi_k[BM];
    __shared__ int32_t seg_cnt[NSEG][BM], seg_off[NSEG][BM], seg_cap[NSEG][BM], seg_ref[NSEG][BM];
    __shared__ int32_t s_head, s_ncols, s_wave[C::NWV];
    __shared__ unsigned long long s_tot_pairs;
    __shared__ int32_t s_tot_rows;
    __shared__ float r_amin[KS][BM], r_bmax[KS][BM];  // relay: per key split, alpha / beta of a row
    __shared__ int32_t r_nc[BM], r_ns[BM];            // relay: the row's ledger counts |R|, |C|
    __shared__ int32_t s_last;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;  // (each tile takes them afresh)
    constexpr int mode = MODE;  // one instance per caller
    const int T = a.k + a.m;
    const int group = a.n_heads / a.n_kv_heads;
    const int n_mand = a.n_sink + a.n_recent;  // mandatory sentinel slots, after the random ones
    const int c_sent = a.m + a.r + n_mand;

    if (a.pairs_out && (mode == MODE_FULL || mode == MODE_ANCHOR) && blockIdx.x == 0 && tid == 0)
        *a.pairs_out = a.pairs_value;

    // Reroute.  With a workgroup for every tile that full routing would have
    // (the grid covers them all), workgroup b owns full routing's tile (h, t):
    // its rows are the head's flagged rows of ranks [t BM, (t+1) BM), found by
    // the flag ranking below (none: the tile is skipped).  Otherwise the
    // workgroups share a per-head tile table (heads in XCD-major order) built
    // from the rescoring workgroups' flagged-row counts.  Wave 0 of workgroup 0
    // also publishes the call's totals (rerouted rows, score pairs).
    int32_t *tb = reinterpret_cast<int32_t *>(smem + a.lds_tiles);
    const int max_tiles = a.n_heads * a.tiles_per_head;
    const bool own_tile = mode == MODE_REROUTE && (int)gridDim.x >= max_tiles;
    if (mode == MODE_REROUTE && !own_tile) {
        for (int j = tid; j < a.n_heads; j += C::NT) {
            const int hd = head_at(j, a.n_heads, a.n_kv_heads);
            const int32_t *bc = a.blk_count + (int64_t)hd * a.rescore_bph;
            // (eight loads in flight at a time)
            int c = 0, b = 0;
            for (; b + 8 <= a.rescore_bph; b += 8) {
                int t8[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) t8[u] = bc[b + u];
#pragma unroll
                for (int u = 0; u < 8; ++u) c += t8[u];
            }
            for (; b < a.rescore_bph; ++b) c += bc[b];
            tb[j + 1] = (c + BM - 1) / BM;
        }
    }
    if (mode == MODE_REROUTE) {
        if (blockIdx.x == 0 && w == 0) {
            // register sums over the rescoring workgroups' counts, four loads
            // of each kind in flight per lane
            unsigned long long pp = 0;
            int cc = 0;
            const int nb = a.n_heads * a.rescore_bph;
            int j = lane;
            for (; j + 192 < nb; j += 256) {
                int64_t p4[4];
                int c4[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    p4[u] = a.blk_pairs[j + 64 * u];
                    c4[u] = a.blk_count[j + 64 * u];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    pp += (unsigned long long)p4[u];
                    cc += c4[u];
                }
            }
            for (; j < nb; j += 64) {
                pp += (unsigned long long)a.blk_pairs[j];
                cc += a.blk_count[j];
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                pp += (unsigned long long)__shfl_xor((long long)pp, off, 64);
                cc += __shfl_xor(cc, off, 64);
            }
            if (lane == 0) {
                *a.stat_pairs = (int64_t)pp;
                *a.stat_nrr = cc;
                if (a.pairs_out) *a.pairs_out = (int64_t)pp;
                if (a.nrr_out) *a.nrr_out = cc;
            }
        }
        if (!own_tile) {
            __syncthreads();
            if (w == 0) {
                // inclusive scan of the heads' tile counts, 64 heads at a time
                int carry = 0;
                for (int j0 = 0; j0 < a.n_heads; j0 += 64) {
                    const int j = j0 + lane;
                    int v = (j < a.n_heads) ? tb[j + 1] : 0;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const int u = __shfl_up(v, off, 64);
                        v += (lane >= off) ? u : 0;
                    }
                    if (j < a.n_heads) tb[j + 1] = v + carry;
                    carry += __shfl(v, 63, 64);
                }
                if (lane == 0) tb[0] = 0;
            }
            __syncthreads();
        }
    }

    // Tiles of this workgroup.  Full / anchor, and reroute with a workgroup
    // per possible tile: one tile per workgroup, mapped XCD-aware.  Other
    // reroutes: the XCD's contiguous range of the tile table (heads in
    // XCD-major order), strided over the XCD's workgroups.
    int tile, t_end, t_step;
    if (mode == MODE_REROUTE && own_tile) {
        tile = blockIdx.x;
        t_step = gridDim.x;
        t_end = tile < max_tiles ? tile + 1 : tile;
    } else if (mode == MODE_REROUTE) {
        if ((a.n_kv_heads & 7) == 0 && (gridDim.x & 7) == 0) {
            const int x = blockIdx.x & 7, hx = a.n_heads >> 3;
            tile = tb[x * hx] + (int)(blockIdx.x >> 3);
            t_end = tb[(x + 1) * hx];
            t_step = gridDim.x >> 3;
        } else {
            tile = blockIdx.x;
            t_end = tb[a.n_heads];
            t_step = gridDim.x;
        }
    } else {
        tile = blockIdx.x;
        t_end = a.n_heads * a.tiles_per_head;
        t_step = gridDim.x;
    }

    for (; tile < t_end; tile += t_step) {
        // the lane's indices are taken afresh on every tile (the empty asm hides
        // where they come from), so that the address arithmetic built on them
        // is recomputed per tile rather than held in registers across the loop
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
        const int rb = w % NW, p = w / NW;
        // ---------------------------------------------------- rows of the tile
        int h, t;
        if (mode == MODE_REROUTE && !own_tile) {
            if (tid == 0) s_head = 0;
            __syncthreads();
            for (int j = tid; j < a.n_heads; j += C::NT)
                if (tb[j] <= tile && tile < tb[j + 1]) s_head = j;
            __syncthreads();
            const int j = s_head;
            h = head_at(j, a.n_heads, a.n_kv_heads);
            t = tile - tb[j];
        } else {
            tile_of_block(tile, a.n_heads, a.n_kv_heads, a.tiles_per_head, h, t);
        }
        // reroute: the flags of the ranking's first pass are requested before
        // the row set-up's barrier
        const uint8_t *fl = a.flags + (int64_t)h * a.n_q;
        bool fpre[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = 4 * tid + j;
            fpre[j] = (mode == MODE_REROUTE) && (i < a.n_q) && fl[i] != 0;
        }
        if (tid < BM) {
            row_g[tid] = -1;
            row_i[tid] = 0;
            row_n[tid] = 0;
        }
        if (tid == 0) s_ncols = 0;
        __syncthreads();
        if (mode == MODE_REROUTE) {
            const int lo = t * BM, hi = lo + BM;
            int run = 0;
            // thread tid takes rows base + 4 tid + j, j < 4 (the four loads in
            // flight together); ranks follow the row order
            for (int base = 0; base < a.n_q && run < hi; base += 4 * C::NT) {
                bool f[4];
                uint64_t mk[4];
                int below = 0, wtot = 0;
                const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int i = base + 4 * tid + j;
                    f[j] = (base == 0) ? fpre[j] : ((i < a.n_q) && fl[i] != 0);
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    mk[j] = __ballot(f[j]);
                    below += __popcll(mk[j] & lt);
                    wtot += __popcll(mk[j]);
                }
                if (lane == 0) s_wave[w] = wtot;
                __syncthreads();
                int pre = run, tot = 0;
#pragma unroll
                for (int v = 0; v < C::NWV; ++v) {
                    pre += (v < w) ? s_wave[v] : 0;
                    tot += s_wave[v];
                }
                int rank = pre + below;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int i = base + 4 * tid + j;
                    if (f[j] && rank >= lo && rank < hi) {
                        row_i[rank - lo] = i;
                        row_g[rank - lo] = h * a.n_q + i;
                    }
                    rank += f[j] ? 1 : 0;
                }
                run += tot;
                __syncthreads();  // (also orders the rows' writes before their reads below)
            }
        } else {
            if (tid < BM) {
                const int i = t * BM + tid;
                if (i < a.n_q) {
                    row_i[tid] = i;
                    row_g[tid] = h * a.n_q + i;
                }
            }
            __syncthreads();
        }
        if (tid < BM) {  // whole waves (BM is 32, or a multiple of 64)
            int rn = 0;
            if (row_g[tid] >= 0) {
                const int i = row_i[tid];
                rn = a.causal ? min(i + 1, a.n_k) : a.n_k;
                row_n[tid] = rn;
                // the row's route width k_i (Sec. 4.3): it selects T_i = k_i + m
                // chunks; the threshold bounds of T = k + m >= T_i stay valid
                row_k[tid] = a.k_rows ? min(max(a.k_rows[row_g[tid]], 1), a.k) : a.k;
            }
            const int m = wave_max_small(rn, 32 - __clz(a.n_k));
            if (lane == 0 && m > 0) atomicMax(&s_ncols, m);
        }
        __syncthreads();
        const int ncols = s_ncols;
        if (ncols == 0) continue;  // no row in this tile (uniform)
        // stages per split and segment length: 2*KS segments of 16*nb keys
        // cover the padded key range
        const int nb = __builtin_amdgcn_readfirstlane((ncols + 32 * KS - 1) / (32 * KS));
        const int seg = 16 * nb;

        const int myrow = 32 * rb + l32;  // this lane's row in the sweeps
        const int nrow = row_n[myrow];
        const int myseg = 2 * p + hh;
        const int sbase = myseg * seg;
        // stages whose keys (up to (2p+1)*seg + 16 st + 15) are valid for every
        // row of the wave
        int minn = (row_g[myrow] >= 0) ? nrow : INT_MAX;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) minn = min(minn, __shfl_xor(minn, off, 64));
        const int slack = minn - (2 * p + 1) * seg - 16;
        const int full_stages = __builtin_amdgcn_readfirstlane(
            (minn == INT_MAX) ? nb : (slack < 0 ? 0 : min(nb, slack / 16 + 1)));
        const unsigned char *Kg =
            reinterpret_cast<const unsigned char *>(a.K) + (int64_t)(h / group) * a.n_k * C::ROWB;
        // relay: the ledger rows -> per-row bitmaps over the key range, (R
        // word, C word) per 32 keys, in the candidate region (free until the
        // collection sweep).  Wave w reads rows w, w + NWV, ..., a lane per
        // ledger slot; every lane loads (masked slots read row 0).  The first
        // chunk of ledger loads and then the query fragments are requested
        // before the bitmap clear, whose barrier orders LDS only, so that
        // both are in flight during it.
        uint2 *rbm = reinterpret_cast<uint2 *>(ss);
        constexpr int RPW = BM / C::NWV;
        static_assert(BM % C::NWV == 0, "rows split evenly over the waves");
        const int c_led = a.k + c_sent;
        int led_id[RPW];
        auto load_led = [&](int s0) __attribute__((always_inline)) {
            const int slot = s0 + lane;
            const bool inr = slot < a.k, live = slot < c_led;
            const int32_t *col = inr ? a.led_routes + slot : (live ? a.led_sent + (slot - a.k) : a.led_routes);
            const int64_t stride = inr ? a.k : (live ? c_sent : a.k);
#pragma unroll
            for (int q = 0; q < RPW; ++q) {
                const int64_t g = row_g[w + q * C::NWV];
                const bool ok = live && g >= 0;
                const int v = col[(ok ? g : 0) * stride];
                led_id[q] = ok ? v : -1;
            }
        };
        if constexpr (mode == MODE_RELAY) load_led(0);

        Frag<DT, D> fq;
        if (row_g[myrow] >= 0)
            fq.load(reinterpret_cast<const DT *>(a.Q) + (int64_t)row_g[myrow] * D, hh);
        else
            fq.zero();

        if constexpr (mode == MODE_RELAY) {
            const int nwd = a.bm_words;
            for (int j = tid; j < BM * nwd; j += C::NT) rbm[j] = make_uint2(0u, 0u);
            if (tid == 0) {
                s_tot_pairs = 0ull;
                s_tot_rows = 0;
            }
            lds_barrier();
            int nc[RPW], ns[RPW];
#pragma unroll
            for (int q = 0; q < RPW; ++q) nc[q] = ns[q] = 0;
            uint32_t *bw = reinterpret_cast<uint32_t *>(rbm);
            for (int s0 = 0; s0 < c_led; s0 += 64) {
                if (s0 > 0) load_led(s0);
                const bool inr = s0 + lane < a.k;
#pragma unroll
                for (int q = 0; q < RPW; ++q) {
                    const int r = w + q * C::NWV;
                    const int id = led_id[q];
                    const bool ok = id >= 0 && id < a.n_k;  // ledger ids lie in [0, n_i); -1 is an empty slot
                    if (ok) atomicOr(&bw[2 * (r * nwd + (id >> 5)) + (inr ? 0 : 1)], 1u << (id & 31));
                    nc[q] += __popcll(__ballot(ok && inr));
                    ns[q] += __popcll(__ballot(ok && !inr));
                }
            }
            if (lane == 0) {
#pragma unroll
                for (int q = 0; q < RPW; ++q) {
                    r_nc[w + q * C::NWV] = nc[q];
                    r_ns[w + q * C::NWV] = ns[q];
                }
            }
            lds_barrier();
        }

        // the collection sweep's key ring; its first two stages are requested
        // as soon as no other sweep needs the loads, so that they arrive
        // during the threshold seeds or the threshold bound
        u32x4_t breg[2][C::PER_T];
        // ------------------------------------------------ sweep 1: thresholds
        if (mode == MODE_REROUTE && a.seed_bound) {
            sweep_db_first<C>(breg, Kg, a.n_k, seg, nb, tid);
            // the rescoring pass scored every key of these rows and left each
            // row's bound and maximum; they are widened by kSeedSlack orders
            // so that they hold even if its scores differ from this tile's in
            // the last bits
            if (tid < BM) {
                const int64_t g = row_g[tid];
                float b = -INFINITY, x = -INFINITY;
                if (g >= 0) {
                    b = a.seed_bound[g];
                    x = a.seed_rmax[g];
                    b = order_float(max(float_order(b) - kSeedSlack, float_order(-INFINITY)));
                    x = order_float(min(float_order(x) + kSeedSlack, float_order(INFINITY)));
                }
                b1_s[tid] = b;
                rmax_s[tid] = x;
            }
        } else if constexpr (mode == MODE_RELAY) {
            {
                RelayEpi<TT> epi;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
#pragma unroll
                    for (int j = 0; j < TT; ++j) epi.top[i][j] = -INFINITY;
                }
                epi.nrow = nrow;
                epi.sbase = sbase;
                epi.amin = INFINITY;
                epi.bmax = -INFINITY;
                epi.bmr = rbm + myrow * a.bm_words;
                epi.wnext = epi.bmr[sbase >> 5];
                sweep_keys<DT, D, C>(fq, Kg, a.n_k, seg, nb, full_stages, tid, p, hh, l32, bt, epi);
                // the row's lanes: halves hh of a wave here, key splits p below
                const float am = fminf(epi.amin, __shfl_xor(epi.amin, 32, 64));
                const float bx = fmaxf(epi.bmax, __shfl_xor(epi.bmax, 32, 64));
                if (hh == 0) {
                    r_amin[p][myrow] = am;
                    r_bmax[p][myrow] = bx;
                }
                __syncthreads();  // every wave is done with the key tiles and the bitmaps
                store_kept<C, TT>(us, myrow, myseg, epi.top);
            }
            __syncthreads();
            sweep_db_first<C>(breg, Kg, a.n_k, seg, nb, tid);
            bound_of_kept<C>(us, tid, T, b1_s, rmax_s);
        } else {
            {
                TopEpi<TT> epi;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
#pragma unroll
                    for (int j = 0; j < TT; ++j) epi.top[i][j] = -INFINITY;
                }
                epi.nrow = nrow;
                epi.sbase = sbase;
                sweep_keys<DT, D, C>(fq, Kg, a.n_k, seg, nb, full_stages, tid, p, hh, l32, bt, epi);
                __syncthreads();  // every wave is done with the key tiles
                store_kept<C, TT>(us, myrow, myseg, epi.top);
            }
            __syncthreads();
            sweep_db_first<C>(breg, Kg, a.n_k, seg, nb, tid);
            bound_of_kept<C>(us, tid, T, b1_s, rmax_s);
        }
        __syncthreads();

        if constexpr (mode == MODE_RELAY) {
            // the trigger (Eq. (8)): a row keeps its route unless C is
            // non-empty and beta + gamma >= alpha.  Kept rows are finished
            // (outputs and age); the rest of the tile routes the flagged rows
            // only, the others now count as padding.  Score pairs follow the
            // method's accounting: the ledger's candidates, plus n_i for each
            // refreshed row.
            unsigned long long pr = 0;
            int cf = 0;
            if (tid < BM && row_g[tid] >= 0) {
                const int64_t row = row_g[tid];
                float al = r_amin[0][tid], be = r_bmax[0][tid];
#pragma unroll
                for (int q = 1; q < KS; ++q) {
                    al = fminf(al, r_amin[q][tid]);
                    be = fmaxf(be, r_bmax[q][tid]);
                }
                const int ncr = r_nc[tid], nsr = r_ns[tid];
                const bool flag = relay_trigger(nsr, al, be, a.gamma, a.gamma_rows, row, a.layer,
                                                a.min_reuse > 0 ? a.led_build[row] : 0, a.min_reuse);
                a.flags[row] = flag ? 1 : 0;
                if (a.mask_out) a.mask_out[row] = flag ? 1 : 0;
                a.alpha_out[row] = al;
                a.beta_out[row] = be;
                if (!flag) {
                    a.led_age[row] = a.layer - a.led_build[row];
                    row_g[tid] = -1;
                }
                pr = (unsigned long long)(ncr + nsr + (flag ? row_n[tid] : 0));
                cf = flag ? 1 : 0;
            }
            if (tid < ((BM + 63) & ~63)) {
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    pr += (unsigned long long)__shfl_xor((long long)pr, off, 64);
                    cf += __shfl_xor(cf, off, 64);
                }
                if (lane == 0) {
                    atomicAdd(&s_tot_pairs, pr);
                    atomicAdd(&s_tot_rows, cf);
                }
            }
            __syncthreads();
            const int tile_flagged = s_tot_rows;
            // the launch's totals: each workgroup publishes its tile's counts
            // and the last one to finish sums them (every relay tile holds a
            // row, so every workgroup gets here exactly once)
            if (tid == 0) {
                a.blk_pairs[blockIdx.x] = (int64_t)s_tot_pairs;
                a.blk_count[blockIdx.x] = s_tot_rows;
                __threadfence();
                s_last = (atomicAdd(a.done, 1u) == gridDim.x - 1) ? 1 : 0;
            }
            __syncthreads();
            if (s_last) {
                __threadfence();
                if (tid == 0) {
                    s_tot_pairs = 0ull;
                    s_tot_rows = 0;
                }
                __syncthreads();
                unsigned long long pp = 0;
                int cc = 0;
                for (int j = tid; j < (int)gridDim.x; j += C::NT) {
                    pp += (unsigned long long)__hip_atomic_load(&a.blk_pairs[j], __ATOMIC_RELAXED,
                                                                __HIP_MEMORY_SCOPE_AGENT);
                    cc += __hip_atomic_load(&a.blk_count[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    pp += (unsigned long long)__shfl_xor((long long)pp, off, 64);
                    cc += __shfl_xor(cc, off, 64);
                }
                if (lane == 0) {
                    atomicAdd(&s_tot_pairs, pp);
                    atomicAdd(&s_tot_rows, cc);
                }
                __syncthreads();
                if (tid == 0) {
                    *a.stat_pairs = (int64_t)s_tot_pairs;
                    *a.stat_nrr = s_tot_rows;
                    if (a.pairs_out) *a.pairs_out = (int64_t)s_tot_pairs;
                    if (a.nrr_out) *a.nrr_out = s_tot_rows;
                    __hip_atomic_store(a.done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            if (tile_flagged == 0) continue;  // (uniform) nothing to route in this tile
        }
        if (tid < BM) {
            const bool real = row_g[tid] >= 0;
            th_s[tid] = real ? b1_s[tid] : INFINITY;  // padding rows collect nothing
            th_id[tid] = INT_MAX;
            rstate[tid] = real ? kSweep : kDone;
            // bisection bounds: b1 admits >= T chunks, nothing reaches past the row maximum
            lo_k[tid] = float_order(b1_s[tid]);
            hi_k[tid] = float_order(rmax_s[tid]) + 1u;
            cnt_hi[tid] = 0;
#pragma unroll
            for (int s = 0; s < NSEG; ++s) {
                seg_off[s][tid] = s * CAPQ;
                seg_cap[s][tid] = real ? CAPQ : 0;
                seg_cnt[s][tid] = 0;
            }
        }
        __syncthreads();

        // ------------------------------------------------ sweep 2: collection
        float *lsA = ss + myrow * C::SS;
        uint16_t *liA = si + myrow * C::SI;
        for (int it = 0;; ++it) {
            {
                CollectEpi epi;
                const int off = seg_off[myseg][myrow];
                epi.th = th_s[myrow];
                epi.th_id = th_id[myrow];
                epi.nrow = nrow;
                epi.sbase = sbase;
                epi.cnt = 0;
                epi.dum = CAPR - off;
                epi.ls = lsA + off;
                epi.li = liA + off;
                if (it > 0) sweep_db_first<C>(breg, Kg, a.n_k, seg, nb, tid);
                sweep_keys_db<DT, D, C>(fq, Kg, a.n_k, seg, nb, full_stages, tid, p, hh, l32, bt, breg, epi);
                if (rstate[myrow] != kDone) seg_cnt[myseg][myrow] = epi.cnt;
            }
            __syncthreads();
            bool again = false;
            if (tid < BM && rstate[tid] != kDone) {
                int total = 0;
                bool fit = true;
#pragma unroll
                for (int s = 0; s < NSEG; ++s) {
                    total += seg_cnt[s][tid];
                    fit = fit && seg_cnt[s][tid] <= seg_cap[s][tid];
                }
                const int Ti = row_k[tid] + a.m;
                const int need = min(Ti, row_n[tid]);
                const float th = th_s[tid];
                // sub-list placements for the next sweep: equal shares of the row
                // region, or the exclusive prefix of a sweep's counts (which then
                // fit exactly when the same threshold is applied again)
                auto place_equal = [&]() {
#pragma unroll
                    for (int s = 0; s < NSEG; ++s) {
                        seg_off[s][tid] = s * CAPQ;
                        seg_cap[s][tid] = CAPQ;
                    }
                };
                auto place_counts = [&](const int32_t (*cnt)[BM]) {
                    int o = 0;
#pragma unroll
                    for (int s = 0; s < NSEG; ++s) {
                        const int c = min(cnt[s][tid], CAPR - o);  // (a placement never leaves the row region)
                        seg_off[s][tid] = o;
                        seg_cap[s][tid] = c;
                        o += c;
                    }
                };
                if (rstate[tid] == kTieCut) {
                    // admitted = cnt_hi + ties with id <= th_id: find the smallest
                    // cut admitting T_i (then exactly T_i: ties come one id at a time)
                    const int mid = th_id[tid];
                    if (total >= Ti) {
                        id_hi[tid] = mid;
#pragma unroll
                        for (int s = 0; s < NSEG; ++s) seg_ref[s][tid] = seg_cnt[s][tid];
                    } else {
                        id_lo[tid] = mid;
                    }
                    const int il = id_lo[tid], ih = id_hi[tid];
                    if (ih - il > 1) {
                        th_id[tid] = il + ((ih - il) >> 1);
                        place_equal();
                        again = true;
                    } else if (mid != ih || !fit) {
                        th_id[tid] = ih;
                        place_counts(seg_ref);  // exactly T_i entries, stored by one more sweep
                        again = true;
                    }
                } else if (total < need) {
                    // fewer than T chunks reach th: th bounds the T-th score from
                    // above; bisect again (adjacent bounds: sweep at lo_k to see
                    // its ties)
                    hi_k[tid] = float_order(th);
                    cnt_hi[tid] = total;
                    const uint32_t lk = lo_k[tid], hk = hi_k[tid];
                    th_s[tid] = order_float(hk - lk > 1u ? lk + ((hk - lk) >> 1) : lk);
                    place_equal();
                    again = true;
                } else if (!fit) {
                    if (total <= CAPR) {
                        place_counts(seg_cnt);  // the same threshold again, every sub-list placed to fit
                    } else {
                        // more candidates than the row region holds: raise the threshold
                        lo_k[tid] = float_order(th);
#pragma unroll
                        for (int s = 0; s < NSEG; ++s) seg_ref[s][tid] = seg_cnt[s][tid];
                        const uint32_t lk = lo_k[tid], hk = hi_k[tid];
                        if (hk - lk > 1u) {
                            th_s[tid] = order_float(lk + ((hk - lk) >> 1));
                        } else {
                            // lo_k is the T-th score: the chunks above it are cnt_hi
                            // < T and the T - cnt_hi lowest ids among its ties
                            // complete the set.  Bisect the id cut between -1 (no
                            // tie) and n_i - 1 (all ties: the sweep just counted).
                            rstate[tid] = kTieCut;
                            id_lo[tid] = -1;
                            id_hi[tid] = row_n[tid] - 1;
                            th_s[tid] = order_float(lk);
                            th_id[tid] = -1 + (row_n[tid] >> 1);
                        }
                        place_equal();
                    }
                    again = true;
                }
                if (!again) {
                    rstate[tid] = kDone;
                    th_s[tid] = INFINITY;  // later sweeps admit nothing for this row
                }
            }
            if (!__syncthreads_or(again ? 1 : 0) || it + 1 >= a.sweep_cap) break;
        }
        // a row still unsettled here stopped at the sweep cap (the bisections
        // need fewer sweeps than the cap, so this does not happen unless the
        // cap is lowered): it is counted for the caller and keeps no
        // candidate, so its entry holds valid ids (R and N empty, sentinels
        // drawn from all valid chunks) instead of a partial list
        if (tid < BM && row_g[tid] >= 0 && rstate[tid] != kDone && a.unconverged) atomicAdd(a.unconverged, 1ull);

        // compact each row's sub-lists into one id-ordered run [0, c): the
        // sub-lists lie in segment order at offsets no lower than the counts
        // before them, so moving entries down in order is safe
        int32_t *rcnt = cnt_hi;  // reused: candidate count per row
        {
            // four lanes per row (as in the selection below), a lane per fourth
            // entry.  Sub-lists only move toward the row start (a placement
            // offset is at least the counts before it), a write lands where
            // an entry at least as early in the same sub-list was read (read
            // before, or by the same instruction), and never in a later
            // sub-list's entries: the moves need no barrier.
            const int r = 16 * w + (lane & 15), qq = lane >> 4;
            if (row_g[r] >= 0) {
                float *rs = ss + r * C::SS;
                uint16_t *ri = si + r * C::SI;
                const bool settled = rstate[r] == kDone;  // (an unsettled row keeps nothing)
                int o = 0;
#pragma unroll
                for (int s = 0; s < NSEG; ++s) {
                    const int c = settled ? min(seg_cnt[s][r], seg_cap[s][r]) : 0;
                    const int from = seg_off[s][r];
                    if (from != o) {
                        for (int j = qq; j < c; j += 4) {
                            const float v = rs[from + j];
                            const uint16_t id = ri[from + j];
                            rs[o + j] = v;
                            ri[o + j] = id;
                        }
                    }
                    o += c;
                }
                if (qq == 0) rcnt[r] = o;
            }
        }
        __syncthreads();

        // ------------------------------------- selection, ledger, sentinels
        // (1) four lanes per row: lane (lane & 15) + 16 qq of wave w serves
        // row 16 w + (lane & 15), quarter qq.  The k-th and T-th scores come
        // from a sorting network over the first NET candidates -- each lane
        // sorts a quarter, two bitonic merge stages across the row's lanes
        // complete it -- then insertion of any further candidates; then each
        // lane takes a quarter of the candidates in id order and stages its R
        // and near-miss (N) entries in LDS (stg, each set in id order, -1
        // padded) at offsets from the counts of the quarters before it.
        static_assert(C::NWV * 16 == BM, "four selection lanes per row fill the workgroup");
        constexpr int QN = NET / 4;
        int32_t *stg = reinterpret_cast<int32_t *>(bt);  // [BM][STG]: R at 0.., N at k..
        int32_t *s_nR = id_lo, *s_nN = id_hi;           // reused: staged R and N counts per row
        {
            const int r = 16 * w + (lane & 15), qq = lane >> 4;
            if (row_g[r] >= 0) {  // the four lanes of a row take this branch together
                const int64_t row = row_g[r];
                const int c = rcnt[r];
                const int ke = min(row_k[r], c), Te = min(row_k[r] + a.m, c);
                const float *rs = ss + r * C::SS;
                const uint16_t *ri = si + r * C::SI;
                float v[QN];
#pragma unroll
                for (int q = 0; q < QN; ++q) {
                    const int e = qq * QN + q;
                    v[q] = (e < c) ? rs[e] : -INFINITY;
                }
                sort_desc<QN>(v);
                // a bitonic split with the partner lane (lane ^ xm) of two
                // descending runs, one taken reversed (rev) or both in place;
                // the upper side keeps the larger of each pair (sixteen
                // independent exchanges: LDS shuffles, which pipeline)
                auto split = [&](int xm, bool upper, bool rev) __attribute__((always_inline)) {
                    if (rev) {
#pragma unroll
                        for (int q = 0; q < QN / 2; ++q) {
                            const float x = v[q], y = v[QN - 1 - q];
                            const float px = __shfl_xor(x, xm, 64), py = __shfl_xor(y, xm, 64);
                            v[q] = upper ? fmaxf(x, py) : fminf(y, px);
                            v[QN - 1 - q] = upper ? fmaxf(y, px) : fminf(x, py);
                        }
                    } else {
#pragma unroll
                        for (int q = 0; q < QN; ++q) {
                            const float px = __shfl_xor(v[q], xm, 64);
                            v[q] = upper ? fmaxf(v[q], px) : fminf(v[q], px);
                        }
                    }
                };
                // quarters 0+1 and 2+3 each sorted over 2 QN, then merged
                split(16, (qq & 1) == 0, true);
                merge_desc<QN>(v);
                split(48, qq < 2, true);
                split(16, (qq & 1) == 0, false);
                merge_desc<QN>(v);
                for (int e = NET; e < c; ++e) {
                    // keep the NET largest (Te <= NET, so the k-th and T-th stay
                    // exact): quarter qq inserts the smaller of x and the last
                    // entry of quarter qq - 1 (the value that quarter evicts)
                    const float x = rs[e];
                    const float pl = __shfl(v[QN - 1], qq > 0 ? lane - 16 : lane, 64);
                    const float xe = qq > 0 ? fminf(x, pl) : x;
                    float prev = v[0];
                    v[0] = fmaxf(prev, xe);
#pragma unroll
                    for (int j = 1; j < QN; ++j) {
                        const float cur = v[j];
                        v[j] = __builtin_amdgcn_fmed3f(prev, cur, xe);
                        prev = cur;
                    }
                }
                // the entry at descending position g, in all four lanes
                auto at_pos = [&](int g) {
                    const int gq = min(max(g, 0) / QN, 3);
                    const float x = sorted_at<QN>(v, min(max(g - qq * QN, 0), QN - 1));
                    return from_row(x, gq);  // (g, hence gq, is the same in the row's lanes)
                };
                // (sum, prefix and position exchanges are dependent chains:
                // row swaps, no LDS round trips)
                auto sum4 = [&](int n) {
                    n += xor16(n, lane);
                    return n + xor32(n, lane);
                };
                // exclusive prefix over the quarters
                auto before = [&](int n) {
                    uint32_t nq[4];
                    rows4((uint32_t)n, nq);
                    return (qq > 0 ? (int)nq[0] : 0) + (qq > 1 ? (int)nq[1] : 0) + (qq > 2 ? (int)nq[2] : 0);
                };
                const float vk = at_pos(ke - 1), vT = at_pos(Te - 1);
                const int gtk = sum4(count_gt<QN>(v, vk)), gtT = sum4(count_gt<QN>(v, vT));
                const int nek = sum4(count_eq<QN>(v, vk)), neT = sum4(count_eq<QN>(v, vT));
                int32_t *sR = stg + r * STG, *sN = sR + a.k;
                float *oS = a.scores_out ? a.scores_out + row * a.k : nullptr;
                // this lane's quarter of the candidates, in id order
                const int qn = (c + 3) >> 2, lo = min(qq * qn, c), hi = min(lo + qn, c);
                // (a tie just past position NET - 1 is invisible in v, hence the
                // last condition)
                const bool unique = nek == 1 && neT == 1 && (c <= NET || Te < NET);
                int nr = 0, nn = 0;
                if (unique && qn <= 16) {
                    // R = {s >= vk}, N = {vT <= s < vk}; the quarter (at most 16
                    // entries, all inside the row region) is read once, every
                    // load in flight together, and both passes run on registers
                    float qs[16];
                    uint16_t qi[16];
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const float x = rs[lo + j];
                        qi[j] = ri[lo + j];
                        qs[j] = (lo + j < hi) ? x : -INFINITY;
                    }
                    bool mR[16], mN[16];
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        mR[j] = qs[j] >= vk;
                        mN[j] = !mR[j] & (qs[j] >= vT);
                        nr += mR[j] ? 1 : 0;
                        nn += mN[j] ? 1 : 0;
                    }
                    int jr = before(nr), jn = before(nn);
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        if (mR[j]) {
                            sR[jr] = qi[j];
                            if (oS) oS[jr] = qs[j];
                        }
                        if (mN[j]) sN[jn] = qi[j];
                        jr += mR[j] ? 1 : 0;
                        jn += mN[j] ? 1 : 0;
                    }
                } else if (unique) {
                    // R = {s >= vk}, N = {vT <= s < vk}
                    for (int e = lo; e < hi; ++e) {
                        const float sc = rs[e];
                        const bool inR = sc >= vk, inN = !inR & (sc >= vT);
                        nr += inR ? 1 : 0;
                        nn += inN ? 1 : 0;
                    }
                    int jr = before(nr), jn = before(nn);
                    for (int e = lo; e < hi; ++e) {
                        const float sc = rs[e];
                        const bool inR = sc >= vk, inN = !inR & (sc >= vT);
                        if (inR) {
                            sR[jr] = ri[e];
                            if (oS) oS[jr] = sc;
                        }
                        if (inN) sN[jn] = ri[e];
                        jr += inR ? 1 : 0;
                        jn += inN ? 1 : 0;
                    }
                } else {
                    // equal scores rank the lower id first: the quarter's entries
                    // equal to vk, and those equal to vT below vk, offset the
                    // ranks of the quarters after it
                    int ek = 0, eT = 0;
                    for (int e = lo; e < hi; ++e) {
                        const float sc = rs[e];
                        ek += (sc == vk) ? 1 : 0;
                        eT += ((sc < vk) & (sc == vT)) ? 1 : 0;
                    }
                    const int ek0 = before(ek), eT0 = before(eT);
                    auto member = [&](float sc, int &eqk, int &eqT, bool &inR, bool &inN) {
                        const bool gk = sc > vk, ekk = sc == vk;
                        const bool gT = sc > vT, eTT = sc == vT;
                        const int rk = gtk + eqk, rT = gtT + eqT;
                        eqk += ekk ? 1 : 0;
                        eqT += (!gk & !ekk & eTT) ? 1 : 0;
                        inR = gk | (ekk & (rk < ke));
                        inN = !inR & ((ekk & (rk < Te)) | (!gk & !ekk & (gT | (eTT & (rT < Te)))));
                    };
                    int eqk = ek0, eqT = eT0;
                    for (int e = lo; e < hi; ++e) {
                        bool inR, inN;
                        member(rs[e], eqk, eqT, inR, inN);
                        nr += inR ? 1 : 0;
                        nn += inN ? 1 : 0;
                    }
                    int jr = before(nr), jn = before(nn);
                    eqk = ek0;
                    eqT = eT0;
                    for (int e = lo; e < hi; ++e) {
                        const float sc = rs[e];
                        bool inR, inN;
                        member(sc, eqk, eqT, inR, inN);
                        if (inR) {
                            sR[jr] = ri[e];
                            if (oS) oS[jr] = sc;
                        }
                        if (inN) sN[jn] = ri[e];
                        jr += inR ? 1 : 0;
                        jn += inN ? 1 : 0;
                    }
                }
                const int tR = sum4(nr), tN = sum4(nn);
                for (int j = tR + qq; j < a.k; j += 4) {
                    sR[j] = -1;
                    if (oS) oS[j] = -INFINITY;
                }
                for (int j = tN + qq; j < a.m; j += 4) sN[j] = -1;
                if (qq == 0) {
                    s_nR[r] = tR;
                    s_nN[r] = tN;
                }
                if (mode != MODE_FULL) {
                    // this row's candidates are consumed (every lane of the row
                    // read its last one above): its bitmap takes their place
                    uint32_t *bmr = reinterpret_cast<uint32_t *>(ss) + r * C::SS;
                    const int nw = (row_n[r] <= 32 * C::BMW) ? (row_n[r] + 31) >> 5 : C::BMW;
                    for (int wd = qq; wd < nw; wd += 4) bmr[wd] = 0u;
                }
            }
        }
        lds_barrier();

        // (2) the workgroup copies the staged rows out (a tile's rows are
        // consecutive in memory except in reroute mode, where each row is
        // still one contiguous run) and marks R u N in the per-row bitmaps.
        // Thread tid visits (r, j) = divmod(tid + i * NT, width), stepped
        // without divisions, four visits at a time: the four rows' indices
        // and staged ids are read from LDS before any of their stores.
        uint32_t *bw = reinterpret_cast<uint32_t *>(ss);
        auto copy_out = [&](int wd, int col0, auto &&put) __attribute__((always_inline)) {
            const int dr = C::NT / wd, dj = C::NT - dr * wd;
            int r = tid / wd, j = tid - r * wd;
            while (r < BM) {
                int rr[4], jj[4], gv[4], iv[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    rr[u] = r;
                    jj[u] = j;
                    r += dr;
                    j += dj;
                    if (j >= wd) {
                        j -= wd;
                        ++r;
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int rc = min(rr[u], BM - 1);  // (visits past the tile read its last row, unused)
                    gv[u] = row_g[rc];
                    iv[u] = stg[rc * STG + col0 + jj[u]];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if ((rr[u] < BM) & (gv[u] >= 0)) put(rr[u], jj[u], (int64_t)gv[u], iv[u]);
            }
        };
        copy_out(a.k, 0, [&](int r, int j, int64_t g, int32_t id) __attribute__((always_inline)) {
            if (a.led_routes) a.led_routes[g * a.k + j] = id;
            if (a.routes_out) a.routes_out[g * a.k + j] = id;
            if (mode != MODE_FULL && id >= 0)
                atomicOr(&bw[r * C::SS + ((id >> 5) & (C::BMW - 1))], 1u << (id & 31));
        });
        if (mode != MODE_FULL) {
            if (a.m > 0) {
                copy_out(a.m, a.k, [&](int r, int j, int64_t g, int32_t id) __attribute__((always_inline)) {
                    a.led_sent[g * c_sent + j] = id;
                    if (id >= 0) atomicOr(&bw[r * C::SS + ((id >> 5) & (C::BMW - 1))], 1u << (id & 31));
                });
            }
            for (int i = tid; i < BM; i += C::NT) {
                const int64_t g = row_g[i];
                if (g >= 0) {
                    a.led_build[g] = a.layer;
                    a.led_age[g] = 0;
                }
            }
            lds_barrier();

            // (3) four lanes per row (lanes l, l+16, l+32, l+48 of a wave, as in
            // the selection): the mandatory and random sentinels
            const int r = 16 * w + (lane & 15), qq = lane >> 4, l16 = lane & 15;
            if (row_g[r] >= 0) {  // the four lanes of a row take this branch together
                const int64_t row = row_g[r];
                const int ni = row_n[r];
                const int nR = s_nR[r], nN = s_nN[r];
                const bool exact_bm = ni <= 32 * C::BMW;
                uint32_t *bmr = bw + r * C::SS;
                const int32_t *lr = stg + r * STG, *ln = lr + a.k;
                // the row's earlier draws, for the exact test past the
                // bitmap's width: in the staging slots after R and N where they fit
                // (read back from the ledger row otherwise)
                int32_t *ldr = stg + r * STG + a.k + a.m;
                const bool draws_in_lds = a.r <= STG - 1 - (a.k + a.m);

                int32_t *out = a.led_sent + row * c_sent + a.m;
                int32_t *mout = out + a.r;  // mandatory slots
                const int32_t *drawn = draws_in_lds ? ldr : out;
                int nM = 0;
                // exact membership of x in R u N u M u {first s draws}: binary
                // searches of the id-sorted staged R and N, then a scan of the
                // (few) mandatory sentinels and of the draws
                auto in_ledger = [&](int x, int s) {
                    int lo = 0, hi = nR;
                    while (lo < hi) {
                        const int md = (lo + hi) >> 1;
                        if (lr[md] < x) lo = md + 1; else hi = md;
                    }
                    if (lo < nR && lr[lo] == x) return true;
                    lo = 0;
                    hi = nN;
                    while (lo < hi) {
                        const int md = (lo + hi) >> 1;
                        if (ln[md] < x) lo = md + 1; else hi = md;
                    }
                    if (lo < nN && ln[lo] == x) return true;
                    for (int q = 0; q < nM; ++q)
                        if (mout[q] == x) return true;
                    for (int q = 0; q < s; ++q)
                        if (drawn[q] == x) return true;
                    return false;
                };
                // mandatory sentinels (Sec. 3.1, item 3): the valid sink chunks
                // [0, n_sink) and recent chunks (the n_recent valid chunks up to
                // the row's position: i when n_q == n_k, else the last key chunk)
                // not in R u N, ascending, into the slots after the random ones;
                // marked, so that the random draws leave them out.  The row's
                // first lane takes them; the others learn the count.
                if (n_mand > 0) {
                    if (qq == 0) {
                        int pos = (a.n_q == a.n_k) ? row_i[r] : a.n_k - 1;
                        pos = min(pos, ni - 1);
                        const int sink_end = min(a.n_sink, ni);
                        const int rec_lo = (a.n_recent > 0) ? max(pos - a.n_recent + 1, sink_end) : pos + 1;
                        auto take = [&](int x) {
                            const bool in_rn = exact_bm ? ((bmr[x >> 5] >> (x & 31)) & 1u) != 0u : in_ledger(x, 0);
                            if (!in_rn) {
                                mout[nM++] = x;
                                atomicOr(&bmr[(x >> 5) & (C::BMW - 1)], 1u << (x & 31));
                            }
                        };
                        for (int x = 0; x < sink_end; ++x) take(x);
                        for (int x = rec_lo; x <= pos; ++x) take(x);
                        for (int q = nM; q < n_mand; ++q) mout[q] = -1;
                    }
                    nM = __shfl(nM, l16, 64);
                }
                // random sentinels: r draws from the valid chunks outside R u N u M
                const int pool = ni - (nR + nN + nM);
                auto marked = [&](int x, int s) {
                    const bool hit = (bmr[(x >> 5) & (C::BMW - 1)] >> (x & 31)) & 1u;
                    return (hit && !exact_bm) ? in_ledger(x, s) : hit;
                };
                // y-th (0-based) chunk of [0, ni) outside R u N u {first s draws}
                auto nth_free = [&](int y, int s) {
                    if (exact_bm) {
                        for (int wd = 0; wd * 32 < ni; ++wd) {
                            const int lim = ni - wd * 32;
                            uint32_t z = ~bmr[wd];
                            if (lim < 32) z &= (1u << lim) - 1u;
                            const int pc = __popc(z);
                            if (y < pc) return wd * 32 + select_bit(z, y);
                            y -= pc;
                        }
                        return -1;
                    }
                    for (int x = 0; x < ni; ++x)
                        if (!in_ledger(x, s) && y-- == 0) return x;
                    return -1;
                };
                const uint64_t h0 = sm64(sm64(sm64(a.seed) ^ (uint64_t)(uint32_t)a.layer) ^ (uint64_t)row);
                // x mod ni by Barrett reduction: hi64(x * M) with
                // M = floor((2^64 - 1) / ni) undershoots the true quotient
                // by at most 1, so at most two corrections remain.  (ni <=
                // n_k <= 8192, so the small-divisor helpers apply.)
                const uint64_t nn = (uint64_t)ni;
                auto mod_ni = [&](uint64_t x, uint64_t M) {
                    uint64_t rm = x - __umul64hi(x, M) * nn;
                    rm = (rm >= nn) ? rm - nn : rm;
                    rm = (rm >= nn) ? rm - nn : rm;
                    return (int)rm;
                };
                if (exact_bm && pool > a.r && 2 * pool > ni) {
                    // Probing with an exact bitmap (the common case): the four
                    // lanes take the slots four at a time.  Each lane hashes its
                    // slot's first probe and reads its bit as the bitmap stands
                    // before the four; then, in slot order, the slot's lane
                    // decides on its first probe, which is also compared with
                    // the choices of the slots before it among the four (not yet
                    // in the bitmap when it was read).  A rejected first probe
                    // is followed by the further probes against the bitmap after
                    // those slots' marks, the lowest attempt that finds its chunk
                    // unmarked winning: by the slot's lane alone where rejections
                    // are rare, four at a time, one per lane, where more than a
                    // quarter of the row's chunks are marked.  The draws are
                    // those of the slots decided one by one.
                    const uint64_t M = max_u64_div_small((uint32_t)ni);
                    const bool coop = 4 * pool < 3 * ni;  // the same in the row's lanes
                    auto bit = [&](int x) { return ((bmr[x >> 5] >> (x & 31)) & 1u) != 0u; };
                    for (int b = 0; b < a.r; b += 4) {
                        const int s = b + qq;
                        const uint64_t hs = sm64(h0 ^ (uint64_t)s);
                        const int x0 = mod_ni(sm64(hs), M);
                        const bool pre = bit(x0);
                        int c0 = -1, c1 = -1, c2 = -1;  // choices of the four's first three slots
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int sq = b + q;  // the slot decided now (the same in the row's lanes)
                            const int first = (pre | (x0 == c0) | (x0 == c1) | (x0 == c2)) ? -1 : x0;
                            int chosen;
                            if (coop) {
                                chosen = __shfl(first, l16 + 16 * q, 64);
                                if ((chosen < 0) & (sq < a.r)) {
                                    const uint64_t hq = sm64(h0 ^ (uint64_t)sq);
                                    for (int at0 = 1; chosen < 0 && at0 < 64; at0 += 4) {
                                        const int at = at0 + qq;
                                        int x = -1;
                                        if (at < 64) {
                                            const int xx = mod_ni(sm64(hq ^ (uint64_t)at), M);
                                            x = bit(xx) ? -1 : xx;
                                        }
                                        const int y0 = __shfl(x, l16, 64), y1 = __shfl(x, l16 + 16, 64);
                                        const int y2 = __shfl(x, l16 + 32, 64), y3 = __shfl(x, l16 + 48, 64);
                                        chosen = y0 >= 0 ? y0 : (y1 >= 0 ? y1 : (y2 >= 0 ? y2 : y3));
                                    }
                                    if (chosen < 0) {
                                        // 64 rejections: the y-th remaining pool chunk, ascending
                                        chosen = nth_free((int)mod_u64_small(sm64(hq ^ 64ull), (uint32_t)(pool - sq)), sq);
                                    }
                                }
                                if ((qq == q) & (sq < a.r)) {
                                    if (chosen >= 0) atomicOr(&bmr[chosen >> 5], 1u << (chosen & 31));
                                    out[sq] = chosen;
                                }
                            } else {
                                chosen = first;
                                if ((qq == q) & (sq < a.r)) {
                                    for (int at = 1; chosen < 0 && at < 64; ++at) {
                                        const int x = mod_ni(sm64(hs ^ (uint64_t)at), M);
                                        if (!bit(x)) chosen = x;
                                    }
                                    if (chosen < 0) {
                                        // 64 rejections: the y-th remaining pool chunk, ascending
                                        chosen = nth_free((int)mod_u64_small(sm64(hs ^ 64ull), (uint32_t)(pool - sq)), sq);
                                    }
                                    if (chosen >= 0) atomicOr(&bmr[chosen >> 5], 1u << (chosen & 31));
                                    out[sq] = chosen;
                                }
                                chosen = __shfl(chosen, l16 + 16 * q, 64);
                            }
                            c0 = (q == 0) ? chosen : c0;
                            c1 = (q == 1) ? chosen : c1;
                            c2 = (q == 2) ? chosen : c2;
                        }
                    }
                } else if (exact_bm && pool > a.r) {
                    // a pool of at most half the valid chunks, exact bitmap:
                    // rank sampling, slot s takes the y-th remaining pool chunk
                    // (ascending), y = probe(s, attempt 0) mod (pool - s).  The y
                    // do not depend on earlier draws: the four lanes hash four
                    // slots at a time, then take the chunks in slot order.
                    for (int b = 0; b < a.r; b += 4) {
                        const int s = b + qq;
                        const int y = (s < a.r) ? (int)mod_u64_small(sm64(sm64(h0 ^ (uint64_t)s)), (uint32_t)(pool - s)) : 0;
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            if ((qq == q) & (s < a.r)) {
                                const int chosen = nth_free(y, s);
                                if (chosen >= 0) atomicOr(&bmr[chosen >> 5], 1u << (chosen & 31));
                                out[s] = chosen;
                            }
                        }
                    }
                } else if (qq == 0) {
                    // the other cases, one lane per row
                    if (pool <= a.r && exact_bm) {
                        // the whole pool, ascending: one pass over the bitmap
                        int s = 0;
                        for (int wd = 0; wd * 32 < ni; ++wd) {
                            const int lim = ni - wd * 32;
                            uint32_t z = ~bmr[wd];
                            if (lim < 32) z &= (1u << lim) - 1u;
                            for (; z != 0u && s < a.r; z &= z - 1u) out[s++] = wd * 32 + __ffs(z) - 1;
                        }
                        for (; s < a.r; ++s) out[s] = -1;
                    } else if (pool <= a.r) {
                        for (int s = 0; s < a.r; ++s) out[s] = (s < pool) ? nth_free(s, 0) : -1;
                    } else if (2 * pool <= ni) {
                        // a pool of at most half the valid chunks: rank sampling,
                        // slot s takes the y-th remaining pool chunk (ascending),
                        // y = probe(s, attempt 0) mod (pool - s)
                        for (int s = 0; s < a.r; ++s) {
                            const uint64_t hs = sm64(h0 ^ (uint64_t)s);
                            const int chosen = nth_free((int)mod_u64_small(sm64(hs), (uint32_t)(pool - s)), s);
                            if (chosen >= 0) atomicOr(&bmr[(chosen >> 5) & (C::BMW - 1)], 1u << (chosen & 31));
                            out[s] = chosen;
                            if (draws_in_lds) ldr[s] = chosen;
                        }
                    } else {
                        // probing past the bitmap's width: a probe's bit is a
                        // filter on the id modulo the width, its hits checked
                        // exactly
                        const uint64_t M = max_u64_div_small((uint32_t)ni);
                        for (int s = 0; s < a.r; ++s) {
                            const uint64_t hs = sm64(h0 ^ (uint64_t)s);
                            // the first probe outside the marked set wins (the
                            // pool holds more than half the valid chunks, so
                            // probe 0 nearly always does)
                            const int x0 = mod_ni(sm64(hs), M);
                            int chosen = marked(x0, s) ? -1 : x0;
                            for (int at = 1; chosen < 0 && at < 64; ++at) {
                                const int x = mod_ni(sm64(hs ^ (uint64_t)at), M);
                                if (!marked(x, s)) chosen = x;
                            }
                            if (chosen < 0) {
                                // 64 rejections: the y-th remaining pool chunk, ascending
                                chosen = nth_free((int)mod_u64_small(sm64(hs ^ 64ull), (uint32_t)(pool - s)), s);
                            }
                            if (chosen >= 0) atomicOr(&bmr[(chosen >> 5) & (C::BMW - 1)], 1u << (chosen & 31));
                            out[s] = chosen;
                            if (draws_in_lds) ldr[s] = chosen;
                        }
                    }
                }
            }
        }
        lds_barrier();
    }
}

template <int MODE, typename DT, int D, int NW, int KS, int TT, int NETW, int CAPQ>
hipError_t launch_t(RouteArgs a, int grid, hipStream_t stream)
{
    using C = RT<DT, D, NW, KS, TT, NETW, CAPQ>;
    const int staging = C::BM * (NETW + 1) * 4;  // R / N staging rows
    const int region0 = ((2 * C::ST > staging ? 2 * C::ST : staging) + 15) & ~15;
    a.lds_region0 = region0;
    size_t lds = (size_t)region0 + (size_t)C::BM * C::SS * 4 + (size_t)C::BM * C::SI * 2;
    static_assert((size_t)C::BM * C::UST * 4 <=
                      (size_t)C::BM * (NETW + 1) * 4 + (size_t)C::BM * C::SS * 4 + (size_t)C::BM * C::SI * 2,
                  "the kept scores of the threshold sweep fit the dynamic region");
    static_assert(MODE != MODE_RELAY || KS == 2,
                  "the relay's bitmap row stride (2 word pairs per 64 keys) covers a key range padded to 64 keys");
    if (MODE == MODE_RELAY && (size_t)a.bm_words * 8 > (size_t)C::SS * 4 + (size_t)C::SI * 2)
        return hipErrorInvalidValue;  // the ledger bitmaps exceed the candidate region
    if (MODE == MODE_REROUTE) {  // the per-head tile table
        lds = (lds + 15) & ~(size_t)15;
        a.lds_tiles = (int32_t)lds;
        lds += (size_t)(a.n_heads + 1) * 4;
    }
    const void *fn = reinterpret_cast<const void *>(&route_kernel<MODE, DT, D, NW, KS, TT, NETW, CAPQ>);
    static LdsLimit seen;
    hipError_t e = raise_lds_limit(fn, lds, seen);
    if (e != hipSuccess) return e;
    if (a.sweep_cap < 1) a.sweep_cap = kMaxFixIters;
    hipLaunchKernelGGL((route_kernel<MODE, DT, D, NW, KS, TT, NETW, CAPQ>), dim3(grid), dim3(64 * NW * KS), lds, stream,
                       a);
    return hipGetLastError();
}

// T = k + m <= 64: 128-row tiles, 8 waves (two key splits), top-2 per slot, a
// 64-entry network; T <= 128: 64-row tiles, 4 waves, top-3, a 128-entry
// network.  The sub-list share CAPQ keeps the workgroup's LDS within 160 KB.
template <typename DT, int D>
using NarrowRT = RT<DT, D, 4, 2, 2, 64, (D * (int)sizeof(DT) <= 256 ? 32 : 20)>;
template <typename DT, int D>
using WideRT = RT<DT, D, 2, 2, 3, 128, (D * (int)sizeof(DT) <= 256 ? 48 : 32)>;
template <typename DT, int D>
using SmallRT = RT<DT, D, 1, 2, 2, 64, (D * (int)sizeof(DT) <= 256 ? 32 : 20)>;

template <int MODE, class C>
hipError_t launch_c(const RouteArgs &a, int grid, hipStream_t stream)
{
    return launch_t<MODE, typename C::DType, C::DIM, C::NW_, C::KS_, C::TT_, C::NET, C::CAPQ_>(a, grid, stream);
}

template <int MODE, typename DT, int D>
hipError_t launch_d(const RouteArgs &a, int grid, hipStream_t stream)
{
    static_assert(WideRT<DT, D>::BM == kWideTileRows && NarrowRT<DT, D>::BM == kNarrowTileRows &&
                      SmallRT<DT, D>::BM == kSmallTileRows,
                  "tile heights of the three classes");
    static_assert(SmallRT<DT, D>::SS == NarrowRT<DT, D>::SS && SmallRT<DT, D>::SI == NarrowRT<DT, D>::SI,
                  "small and narrow tiles give a row the same candidate region");
    if (a.k + a.m > 64) return launch_c<MODE, WideRT<DT, D>>(a, grid, stream);
    if (a.tile_rows == kSmallTileRows) return launch_c<MODE, SmallRT<DT, D>>(a, grid, stream);
    return launch_c<MODE, NarrowRT<DT, D>>(a, grid, stream);
}

// Ledger bitmap words (R, C pairs per row) that a relay tile's candidate
// region holds.
template <typename DT, int D>
int relay_max_bm_words(int T)
{
    if (T > 64) return (WideRT<DT, D>::SS * 4 + WideRT<DT, D>::SI * 2) / 8;
    return (NarrowRT<DT, D>::SS * 4 + NarrowRT<DT, D>::SI * 2) / 8;
}

template <int MODE, typename DT>
hipError_t launch_family(const RouteArgs &a, int grid, hipStream_t stream)
{
    switch (a.d) {
    case 32: return launch_d<MODE, DT, 32>(a, grid, stream);
    case 64: return launch_d<MODE, DT, 64>(a, grid, stream);
    case 128: return launch_d<MODE, DT, 128>(a, grid, stream);
    case 256:
        if constexpr (sizeof(DT) == 2) return launch_d<MODE, DT, 256>(a, grid, stream);
        break;
    default: break;
    }
    return hipErrorInvalidValue;
}

}  // namespace route_detail
}  // namespace rr
