// Device helpers of the gfx950 route-maintenance kernels: operand fragments
// for the 32x32 MFMA tiles, the total rank order of (score, chunk id), wave
// shuffles and the random-probe counter hash.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rr {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Storage tag of bf16 inputs (the bits are read as __bf16 vectors).
// Four 32-bit lanes loaded or stored as one 16-byte vector (a native vector
// type, so arrays of them stay in registers).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

struct bf16_t {
    uint16_t bits;
};

// ---------------------------------------------------------------- ordering
//
// Rank order: a higher score ranks first; equal scores rank the lower chunk
// id first; -0 and +0 are the same score.  rank_key maps (score, id) to a
// 64-bit integer that is larger exactly when the pair ranks earlier, so all
// keys of a row are distinct.

__device__ __forceinline__ uint32_t float_order(float s)
{
    uint32_t b = __float_as_uint(s);
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float order_float(uint32_t o)
{
    uint32_t b = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(b);
}

__device__ __forceinline__ uint64_t rank_key(float s, int32_t id)
{
    return ((uint64_t)float_order(s) << 32) | (uint64_t)(uint32_t)(~id);
}

__device__ __forceinline__ int32_t key_id(uint64_t key) { return (int32_t)(~(uint32_t)key); }

__device__ __forceinline__ float key_score(uint64_t key) { return order_float((uint32_t)(key >> 32)); }

// ---------------------------------------------------------------- shuffles

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src)
{
    uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, 64);
    uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, 64);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask)
{
    uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, mask, 64);
    uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), mask, 64);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t lanemask_lt32(int l32) { return (1u << l32) - 1u; }

// ------------------------------------------------------------ trigger
//
// Eq. (8): a row keeps its route while alpha > beta + gamma_i.  It is
// rerouted when it has a sentinel, its minimum reuse horizon has passed
// (Sec. 3.2, Hysteresis: a row (re)built at layer b keeps its route at
// layers b+1 .. b+min_reuse; 0 disables it) and beta + gamma_i >= alpha.
// gamma_i is gamma_rows[row] when the caller gives per-row margins.
__device__ __forceinline__ bool relay_trigger(int n_sent, float alpha, float beta, float gamma,
                                              const float *gamma_rows, int64_t row, int layer, int build,
                                              int min_reuse)
{
    const float g = gamma_rows ? gamma_rows[row] : gamma;
    const bool settled = min_reuse > 0 && layer - build <= min_reuse;
    return n_sent > 0 && !settled && (beta + g >= alpha);
}

// ------------------------------------------------------------ probe hash
//
// splitmix64 output function (Steele, Lea and Flood, OOPSLA 2014): add the
// golden-ratio increment, two xor-shift-multiply rounds, a final xor-shift.
// A random-sentinel probe hashes (seed, layer, row, slot, attempt) by mixing
// each coordinate in with xor and applying the function again.

__device__ __forceinline__ uint64_t sm64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// (The next three are host functions as well, so that a host program can
// check them against exact integer arithmetic.)
//
// x mod m for 0 < m < 2^16, exactly the 64-bit remainder: long division in
// 16-bit digits, where each partial remainder (< m) times 2^16 plus the next
// digit stays below 2^32, so four 32-bit remainders replace the 64-bit one.
__host__ __device__ __forceinline__ uint32_t mod_u64_small(uint64_t x, uint32_t m)
{
    uint32_t r = (uint32_t)(x >> 48) % m;
    r = ((r << 16) | (uint32_t)((x >> 32) & 0xffffu)) % m;
    r = ((r << 16) | (uint32_t)((x >> 16) & 0xffffu)) % m;
    return ((r << 16) | (uint32_t)(x & 0xffffu)) % m;
}

// floor((2^64 - 1) / m) for 0 < m < 2^16, by the same 16-bit long division
__host__ __device__ __forceinline__ uint64_t max_u64_div_small(uint32_t m)
{
    uint64_t q = 0;
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t cur = (r << 16) | 0xffffu;
        q = (q << 16) | (uint64_t)(cur / m);
        r = cur % m;
    }
    return q;
}

// x of lane (lane ^ 1), resp. (lane ^ 2), within each group of four lanes:
// DPP quad permutations [1,0,3,2] and [2,3,0,1] (a VALU move, where a shuffle
// through ds_bpermute takes an LDS round trip).  Every lane must be active.
__device__ __forceinline__ int quad_xor1(int x) { return __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false); }
__device__ __forceinline__ int quad_xor2(int x) { return __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false); }
__device__ __forceinline__ float quad_xor1(float x) { return __int_as_float(quad_xor1(__float_as_int(x))); }
__device__ __forceinline__ float quad_xor2(float x) { return __int_as_float(quad_xor2(__float_as_int(x))); }

// Exchanges among the four lanes l16 + 16 q (q = 0..3, l16 = lane & 15) of a
// wave, by gfx950's row swaps.  With both operands x, v_permlane16_swap
// yields x of lanes l & ~16 and l | 16, v_permlane32_swap x of lanes l & ~32
// and l | 32.  A lane's partners (its lane ^ 16, lane ^ 32) must be active.
// Each swap costs two copies (it overwrites both operands), a wait state and
// a select: it shortens a chain of dependent exchanges, where a shuffle
// through ds_bpermute waits an LDS round trip each time, but many
// independent exchanges pipeline better as shuffles.
__device__ __forceinline__ void rows4(uint32_t x, uint32_t (&n)[4])
{
    const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);        // x[l & ~16], x[l | 16]
    const auto a = __builtin_amdgcn_permlane32_swap(p[0], p[0], false, false);  // x[l16], x[l16 + 32]
    const auto b = __builtin_amdgcn_permlane32_swap(p[1], p[1], false, false);  // x[l16 + 16], x[l16 + 48]
    n[0] = a[0];
    n[1] = b[0];
    n[2] = a[1];
    n[3] = b[1];
}
// x of lane l16 + 16 q, for q the same in the four lanes
__device__ __forceinline__ uint32_t from_row(uint32_t x, int q)
{
    const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    const uint32_t h = (q & 1) ? p[1] : p[0];
    const auto a = __builtin_amdgcn_permlane32_swap(h, h, false, false);
    return (q & 2) ? a[1] : a[0];
}
__device__ __forceinline__ float from_row(float x, int q) { return __uint_as_float(from_row(__float_as_uint(x), q)); }
__device__ __forceinline__ uint32_t xor16(uint32_t x, int lane)
{
    const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return (lane & 16) ? p[0] : p[1];
}
__device__ __forceinline__ uint32_t xor32(uint32_t x, int lane)
{
    const auto p = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return (lane & 32) ? p[0] : p[1];
}
__device__ __forceinline__ int xor16(int x, int lane) { return (int)xor16((uint32_t)x, lane); }
__device__ __forceinline__ int xor32(int x, int lane) { return (int)xor32((uint32_t)x, lane); }

// Largest v over the wave's active lanes, for 0 <= v < 2^nbits, wave-uniform:
// the bits of the maximum from the top, one ballot each.  (An atomic max from
// every lane compiles to a loop over the active lanes, one at a time.)
__device__ __forceinline__ int wave_max_small(int v, int nbits)
{
    int m = 0;
    for (int b = nbits - 1; b >= 0; --b) {
        const int c = m | (1 << b);
        m = (__ballot(v >= c) != 0ull) ? c : m;
    }
    return m;
}

// Position of the y-th (0-based) set bit of z, for y < popc(z): a binary
// search on the population counts of the lower halves.
__host__ __device__ __forceinline__ int select_bit(uint32_t z, int y)
{
    int pos = 0;
#pragma unroll
    for (int wdt = 16; wdt > 0; wdt >>= 1) {
        const uint32_t lo = z & ((1u << wdt) - 1u);
        const int c = __builtin_popcount(lo);
        const bool up = y >= c;
        y = up ? y - c : y;
        z = up ? (z >> wdt) : lo;
        pos = up ? pos + wdt : pos;
    }
    return pos;
}

// Workgroup barrier that orders LDS only: it waits for this wave's LDS
// operations but not for its outstanding global stores, which no thread of
// the workgroup reads back.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// --------------------------------------------------------------- fragments
//
// One lane of a 32x32 MFMA holds, for its row (A) or column (B) lane%32, the
// contiguous half [hh*D/2, (hh+1)*D/2) of the d-dimension, hh = lane/32.  A
// and B use the same split, so every product pairs equal d-indices and the
// sum over the whole d-range is the score.

template <typename DT, int D>
struct Frag;

template <int D>
struct Frag<float, D> {
    static constexpr int NS = D / 2;  // v_mfma_f32_32x32x2_f32 steps
    float v[NS];

    __device__ __forceinline__ void load(const float *row, int hh)
    {
        const float4 *p = reinterpret_cast<const float4 *>(row + hh * (D / 2));
#pragma unroll
        for (int j = 0; j < D / 8; ++j) {
            float4 x = p[j];
            v[4 * j + 0] = x.x;
            v[4 * j + 1] = x.y;
            v[4 * j + 2] = x.z;
            v[4 * j + 3] = x.w;
        }
    }

    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int s = 0; s < NS; ++s) v[s] = 0.f;
    }

    __device__ __forceinline__ static f32x16_t mma(const Frag &a, const Frag &b, f32x16_t c)
    {
#pragma unroll
        for (int s = 0; s < NS; ++s) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[s], b.v[s], c, 0, 0, 0);
        return c;
    }

    // step s of the product (s a compile-time constant after unrolling)
    __device__ __forceinline__ static f32x16_t mma_step(const Frag &a, const Frag &b, f32x16_t c, int s)
    {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[s], b.v[s], c, 0, 0, 0);
    }
};

template <int D>
struct Frag<bf16_t, D> {
    static constexpr int NS = D / 16;  // v_mfma_f32_32x32x16_bf16 steps
    bf16x8_t v[NS];

    __device__ __forceinline__ void load(const bf16_t *row, int hh)
    {
        const bf16x8_t *p = reinterpret_cast<const bf16x8_t *>(row + hh * (D / 2));
#pragma unroll
        for (int j = 0; j < NS; ++j) v[j] = p[j];
    }

    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[s][e] = (__bf16)0.0f;
        }
    }

    __device__ __forceinline__ static f32x16_t mma(const Frag &a, const Frag &b, f32x16_t c)
    {
#pragma unroll
        for (int s = 0; s < NS; ++s) c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v[s], b.v[s], c, 0, 0, 0);
        return c;
    }

    // step s of the product (s a compile-time constant after unrolling)
    __device__ __forceinline__ static f32x16_t mma_step(const Frag &a, const Frag &b, f32x16_t c, int s)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v[s], b.v[s], c, 0, 0, 0);
    }
};

// Workgroup-to-(head, tile) map.  With a multiple of 8 key heads, the tiles
// of key head g go to workgroups b with b % 8 == g % 8: workgroups are handed
// to the 8 XCDs round-robin, so each XCD's L2 serves the key rows of its own
// heads only.
__device__ __forceinline__ void tile_of_block(int b, int H, int Hkv, int tph, int &h, int &t)
{
    const int group = H / Hkv;
    if ((Hkv & 7) == 0) {
        const int x = b & 7, local = b >> 3;
        const int j = local / tph;
        t = local - j * tph;
        const int g = x + 8 * (j / group);
        h = g * group + (j - (j / group) * group);
    } else {
        h = b / tph;
        t = b - h * tph;
    }
}

// Query head at position j of the XCD-major head order: with a multiple of 8
// key heads, positions [x*H/8, (x+1)*H/8) hold the query heads whose key head
// g has g % 8 == x, so per-XCD work lists are contiguous.
__device__ __forceinline__ int head_at(int j, int H, int Hkv)
{
    if ((Hkv & 7) != 0) return j;
    const int group = H / Hkv, hx = H >> 3;
    const int x = j / hx, local = j - x * hx;
    const int g = x + 8 * (local / group);
    return g * group + (local - (local / group) * group);
}

// Row of the 32x32 accumulator held in register i by a lane of half hh.
__device__ __forceinline__ int acc_row(int i, int hh) { return 8 * (i >> 2) + 4 * hh + (i & 3); }

}  // namespace rr
