// The steps either side of route maintenance, for gfx950:
//
//  * chunk pooling (Sec. 2.1): one representation per chunk of tokens, the
//    mean of its token vectors -- a streaming pass at HBM rate;
//  * token expansion (Sec. 2.1): routed chunk ids -> token ids;
//  * sparse attention over the routed chunks' tokens (Sec. 2.2 Eq. (3)): a
//    flash-style kernel on bf16 MFMA tiles with an online softmax.
//
// Sparse attention.  A workgroup takes up to 256 query tokens of one query
// chunk (8 waves of 32 queries, one head) and walks the route of that chunk:
// each routed chunk is cut into 64-key sub-blocks, staged in LDS (K and V
// row-major, loaded a key row per 16 lanes) with the next sub-block's global
// loads in flight during the current one's products.  Per 32-key block a
// wave computes S^T = K Q^T (keys x queries, so every lane owns one query),
// applies the mask and the online-softmax update in registers, and
// accumulates O^T = V^T P^T with P taken straight from the S^T accumulator:
// the keys of the PV product are ordered the way the accumulator holds them
// (each lane half holds groups of 4 consecutive keys, 8 apart), and the V^T
// operand is read from the row-major V tile with the LDS transpose read.
#include <hip/hip_runtime.h>

#include <cmath>

#include "rr_device.hpp"
#include "rr_internal.hpp"

namespace rr {
namespace {

__device__ __forceinline__ float bf16_to_float(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// binary32 -> bf16, round to nearest, ties to even (inputs are finite)
__device__ __forceinline__ uint16_t float_to_bf16(float x)
{
    const uint32_t b = __float_as_uint(x);
    return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// ------------------------------------------------------------- pooling

constexpr int kPoolThreads = 256;

// One workgroup per (head, chunk).  Thread (token lane tl, group g) sums VEC
// consecutive features of tokens tl, tl + TL, ... of the chunk in binary32;
// the TL partial sums of each feature are then added in LDS and divided by
// the chunk's length.
template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const T *__restrict__ X, int n_tok, int d, int chunk,
                                                            int nc, T *__restrict__ out)
{
    constexpr int VEC = 16 / (int)sizeof(T);
    extern __shared__ float part[];  // [TL][d]
    const int hj = blockIdx.x, h = hj / nc, j = hj - h * nc;
    const int G = d / VEC, TL = kPoolThreads / G;
    const int tid = threadIdx.x, tl = tid / G, g = tid - tl * G;
    const int lo = j * chunk, hi = min(lo + chunk, n_tok), len = hi - lo;
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    if (tl < TL) {
        const T *base = X + ((int64_t)h * n_tok + lo) * d + g * VEC;
        for (int t = tl; t < len; t += TL) {
            const u32x4_t v = *reinterpret_cast<const u32x4_t *>(base + (int64_t)t * d);
            if constexpr (sizeof(T) == 4) {
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] += __uint_as_float(v[e]);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] += bf16_to_float((uint16_t)(v[e] & 0xFFFFu));
                    acc[2 * e + 1] += bf16_to_float((uint16_t)(v[e] >> 16));
                }
            }
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) part[tl * d + g * VEC + e] = acc[e];
    }
    __syncthreads();
    for (int f = tid; f < d; f += kPoolThreads) {
        float s = 0.f;
        for (int q = 0; q < TL; ++q) s += part[q * d + f];
        const float mean = s / (float)len;
        T *o = out + ((int64_t)h * nc + j) * d + f;
        if constexpr (sizeof(T) == 4)
            *o = mean;
        else
            o->bits = float_to_bf16(mean);
    }
}

// ------------------------------------------------------------ expansion

__global__ void expand_kernel(const int32_t *__restrict__ routes, int64_t rows, int k, int chunk, int n_tok,
                              int32_t *__restrict__ tokens)
{
    const int nc = (n_tok + chunk - 1) / chunk;
    const int64_t per_row = (int64_t)k * chunk, total = rows * per_row;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = x / per_row;
        const int c = (int)(x - r * per_row), s = c / chunk, t = c - s * chunk;
        const int j = routes[r * k + s];
        const int64_t u = (int64_t)j * chunk + t;
        tokens[x] = (j >= 0 && j < nc && u < n_tok) ? (int32_t)u : -1;
    }
}

// ------------------------------------------------------ sparse attention

constexpr int kQT = 256;            // query tokens per workgroup
constexpr int kQB = 1;              // 32-query blocks per wave (each K / V operand read feeds kQB products)
constexpr int kAW = kQT / (32 * kQB);  // waves (two per SIMD)
constexpr int kAT = 64 * kAW;       // threads
constexpr int kKB = 64;             // keys per staged sub-block
constexpr float kLazy = 8.f;        // log2 headroom of the running softmax maximum

template <int D>
struct AttnShape {
    static constexpr int KRS = 2 * D + 16;           // bytes per row of the K tile
    // bytes per row of the V tile: the transposed reads of 16 lanes cover 4
    // rows x 32 bytes, which this stride places in distinct banks for the 32
    // lanes served together
    static constexpr int VRS = 2 * D + 64;
    static constexpr int KBYTES = kKB * KRS;          // K tile
    static constexpr int VBYTES = kKB * VRS;          // V tile (row-major like K)
    static constexpr int BUF = KBYTES + VBYTES;       // one stage
    static constexpr int LDS = 2 * BUF;               // double-buffered
    static constexpr int ITEMS = kKB * (D / 8);       // 16-byte pieces of K (and of V) per sub-block
    static constexpr int PT = (ITEMS + kAT - 1) / kAT;
};

typedef short short4_t __attribute__((ext_vector_type(4)));

// Four bf16 of a transposed LDS read (ds_read_b64_tr_b16): lane i of each
// 16-lane group receives element i % 4 of the 8 bytes that lane 4e + i / 4 of
// its group addresses, as element e.
__device__ __forceinline__ short4_t lds_read_tr16(const unsigned char *p)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t *)p);
}

// One sub-block's staging registers: its K and V pieces (consecutive lanes
// read one key row).
template <int D>
struct Stage {
    u32x4_t k[AttnShape<D>::PT], v[AttnShape<D>::PT];

    __device__ __forceinline__ void load(const bf16_t *Kh, const bf16_t *Vh, int u0, int u1, int tid)
    {
        using S = AttnShape<D>;
        const u32x4_t z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int q = 0; q < S::PT; ++q) {
            const int it = tid + q * kAT, grp = it % (D / 8), key = it / (D / 8);
            const bool ok = it < S::ITEMS && u0 + key < u1;
            const int64_t off = (int64_t)(u0 + key) * D + 8 * grp;
            k[q] = ok ? *reinterpret_cast<const u32x4_t *>(Kh + off) : z;
            v[q] = ok ? *reinterpret_cast<const u32x4_t *>(Vh + off) : z;
        }
    }

    __device__ __forceinline__ void store(unsigned char *buf, int tid) const
    {
        using S = AttnShape<D>;
        unsigned char *vt = buf + S::KBYTES;
#pragma unroll
        for (int q = 0; q < S::PT; ++q) {
            const int it = tid + q * kAT, grp = it % (D / 8), key = it / (D / 8);
            if (it < S::ITEMS) {
                *reinterpret_cast<u32x4_t *>(buf + key * S::KRS + 16 * grp) = k[q];
                *reinterpret_cast<u32x4_t *>(vt + key * S::VRS + 16 * grp) = v[q];
            }
        }
    }
};

// Cursor over the (chunk, sub-block) sequence of a workgroup's route.
struct Cursor {
    int ci, sb;
};

template <int D>
__global__ __launch_bounds__(kAT) void sparse_attention_kernel(AttnArgs a)
{
    using S = AttnShape<D>;
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int32_t s_chunk[kMaxAttnSlots];
    __shared__ int32_t s_wcnt[kAW];
    __shared__ int32_t s_n;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
    const int group = a.n_heads / a.n_kv_heads;
    // workgroup -> (key head g, query chunk i, query head within the group, query tile)
    int b = blockIdx.x;
    const int qt = b % a.tiles_per_chunk;
    b /= a.tiles_per_chunk;
    const int hl = b % group;
    b /= group;
    const int i = b % a.n_chunks, g = b / a.n_chunks;
    const int h = g * group + hl;
    const int c_lo = i * a.chunk, c_hi = min(c_lo + a.chunk, a.n_tokens);
    const int q_lo = c_lo + qt * kQT, q_hi = min(q_lo + kQT, c_hi);
    if (q_lo >= q_hi) return;  // (uniform) a tile past a short last chunk

    // the route's admissible chunks, in slot order (ballot compaction)
    const int64_t row = (int64_t)h * a.n_chunks + i;
    if (tid == 0) s_n = 0;
    __syncthreads();
    for (int s0 = 0; s0 < a.k; s0 += kAT) {
        const int s = s0 + tid;
        int j = -1;
        if (s < a.k) j = a.routes[row * a.k + s];
        const bool ok = s < a.k && j >= 0 && j < a.n_chunks && (!a.causal || j <= i);
        const uint64_t mk = __ballot(ok);
        if (lane == 0) s_wcnt[w] = __popcll(mk);
        __syncthreads();
        int pre = s_n;
        for (int v = 0; v < w; ++v) pre += s_wcnt[v];
        if (ok) s_chunk[pre + __popcll(mk & ((1ull << lane) - 1ull))] = j;
        __syncthreads();
        if (tid == 0) {
            int t = 0;
            for (int v = 0; v < kAW; ++v) t += s_wcnt[v];
            s_n += t;
        }
        __syncthreads();
    }
    const int n_ch = s_n;

    // key range [u0, u1) of sub-block sb of admissible chunk ci
    auto range = [&](const Cursor &c, int &u0, int &u1) {
        const int j = s_chunk[c.ci];
        const int k_lo = j * a.chunk;
        int k_hi = min(k_lo + a.chunk, a.n_tokens);
        if (a.causal && j == i) k_hi = min(k_hi, q_hi);  // keys past the tile's last query see no query
        u0 = k_lo + c.sb * kKB;
        u1 = min(u0 + kKB, k_hi);
    };
    auto advance = [&](Cursor &c) {
        int u0, u1;
        range(c, u0, u1);
        const int j = s_chunk[c.ci];
        int k_hi = min(j * a.chunk + a.chunk, a.n_tokens);
        if (a.causal && j == i) k_hi = min(k_hi, q_hi);
        if (u1 >= k_hi) {
            ++c.ci;
            c.sb = 0;
        } else {
            ++c.sb;
        }
    };

    const int t0 = q_lo + 32 * kQB * w;  // this wave's first query
    const bool wave_on = t0 < q_hi;
    const bf16_t *Qg = static_cast<const bf16_t *>(a.Q);
    Frag<bf16_t, D> fq[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        const int t = t0 + 32 * qb + l32;
        if (t < q_hi)
            fq[qb].load(Qg + ((int64_t)h * a.n_tokens + t) * D, hh);
        else
            fq[qb].zero();
    }
    const float c2 = a.scale * 1.4426950408889634f;  // scores in log2 units

    constexpr int NMB = D / 32;
    f32x16_t o[kQB][NMB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
#pragma unroll
            for (int r = 0; r < 16; ++r) o[qb][mb][r] = 0.f;
        }
    }
    float m_run[kQB], l_run[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        m_run[qb] = -INFINITY;
        l_run[qb] = 0.f;
    }

    const bf16_t *Kh = static_cast<const bf16_t *>(a.K) + (int64_t)g * a.n_tokens * D;
    const bf16_t *Vh = static_cast<const bf16_t *>(a.V) + (int64_t)g * a.n_tokens * D;
    Stage<D> st;
    Cursor cur{0, 0};
    if (n_ch > 0) {
        int u0, u1;
        range(cur, u0, u1);
        st.load(Kh, Vh, u0, u1, tid);
        st.store(smem, tid);
    }
    __syncthreads();

    for (int it = 0; cur.ci < n_ch; ++it) {
        int u0, u1;
        range(cur, u0, u1);
        Cursor nxt = cur;
        advance(nxt);
        const bool more = nxt.ci < n_ch;
        if (more) {
            int v0, v1;
            range(nxt, v0, v1);
            st.load(Kh, Vh, v0, v1, tid);
        }
        const unsigned char *buf = smem + (it & 1) * S::BUF;
        const unsigned char *vt = buf + S::KBYTES;
#pragma unroll
        for (int kb = 0; kb < kKB / 32; ++kb) {
            const int k0 = u0 + 32 * kb;
            // (wave-uniform) keys of this block exist and some reach a query of the wave
            if (!wave_on || k0 >= u1 || (a.causal && k0 > t0 + 32 * kQB - 1)) continue;
            // S^T = K Q^T for the wave's query blocks: each K operand feeds kQB products
            f32x16_t sc[kQB];
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb) sc[qb] = f32x16_t{};
#pragma unroll
            for (int q = 0; q < D / 16; ++q) {
                const bf16x8_t kf =
                    *reinterpret_cast<const bf16x8_t *>(buf + (32 * kb + l32) * S::KRS + hh * D + 16 * q);
#pragma unroll
                for (int qb = 0; qb < kQB; ++qb)
                    sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, fq[qb].v[q], sc[qb], 0, 0, 0);
            }
            // (wave-uniform) no key of the block is masked for any query of the wave
            const bool open = k0 + 31 < u1 && (!a.causal || k0 + 31 <= t0);
            bf16x8_t pb[kQB][2];
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb) {
                // mask, then the online-softmax update of this lane's query.  The
                // running maximum m (in log2 units) moves only when a score
                // exceeds it by more than kLazy, so the rescaling of O and l
                // (one multiply per accumulator) is rare; weights are then at
                // most 2^kLazy, and the normalised result is the same
                if (!open) {  // (wave-uniform) key u is admissible iff u <= lim
                    const int t = t0 + 32 * qb + l32;
                    const int lim = a.causal ? min(u1 - 1, t) : u1 - 1;
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        sc[qb][r] = (k0 + acc_row(r, hh) <= lim) ? sc[qb][r] : -INFINITY;
                }
                float mx = sc[qb][0];
#pragma unroll
                for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sc[qb][r]);
                mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c2;
                const bool bump = mx > m_run[qb] + kLazy;
                if (__ballot(bump) != 0ull) {  // (wave-uniform) some query of the wave moves its maximum
                    const float m_new = bump ? mx : m_run[qb];
                    const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);  // 0 from -inf, 1 if unmoved
                    l_run[qb] *= alpha;
#pragma unroll
                    for (int mb = 0; mb < NMB; ++mb) {
#pragma unroll
                        for (int r = 0; r < 16; ++r) o[qb][mb][r] *= alpha;
                    }
                    m_run[qb] = m_new;
                }
                const float m_use = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
                float ls = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    // (v_exp_f32 flushes results below 2^-126 to zero: weights that small vanish
                    // in the binary32 sums anyway)
                    const float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][r], c2, -m_use));
                    ls += pr;
                    pb[qb][r >> 3][r & 7] = (__bf16)pr;
                }
                l_run[qb] += ls;
            }
            // O^T += V^T P^T: each V operand feeds kQB products
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb) {
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    // the A operand of lane (feature 32 mb + l32, half hh): keys
                    // k0 .. k0+3 and k0+8 .. k0+11 of the block, k0 = 16 s2 + 4 hh,
                    // the order in which the accumulator holds this half's keys
                    // (rows 8*(i>>2) + 4*hh + (i&3) of register i); two transposed
                    // reads, lane j of each 16-lane group addressing key row
                    // k0 + j/4 at features 16*(l32/16) + 4*(j%4) of the block
                    const int j = lane & 15;
                    const unsigned char *vp = vt + (32 * kb + 16 * s2 + 4 * hh + (j >> 2)) * S::VRS +
                                              2 * (32 * mb + 16 * (l32 >> 4) + 4 * (j & 3));
                    const short4_t lo = lds_read_tr16(vp), hi = lds_read_tr16(vp + 8 * S::VRS);
                    const bf16x8_t vf = __builtin_bit_cast(
                        bf16x8_t, (short __attribute__((ext_vector_type(8)))){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
                    for (int qb = 0; qb < kQB; ++qb)
                        o[qb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[qb][s2], o[qb][mb], 0, 0, 0);
                }
            }
        }
        if (more) st.store(smem + ((it + 1) & 1) * S::BUF, tid);
        __syncthreads();
        cur = nxt;
    }

    // normalise and write each query row (4 consecutive features per store);
    // the two lane halves of a query hold the partial sums of l
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        const int t = t0 + 32 * qb + l32;
        const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32, 64);
        if (t < q_hi) {
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            bf16_t *orow = static_cast<bf16_t *>(a.O) + ((int64_t)h * a.n_tokens + t) * D;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int f = 32 * mb + 8 * q + 4 * hh;
                    const f32x16_t &ov = o[qb][mb];
                    uint2 pk;
                    pk.x = (uint32_t)float_to_bf16(ov[4 * q] * inv) | ((uint32_t)float_to_bf16(ov[4 * q + 1] * inv) << 16);
                    pk.y = (uint32_t)float_to_bf16(ov[4 * q + 2] * inv) | ((uint32_t)float_to_bf16(ov[4 * q + 3] * inv) << 16);
                    *reinterpret_cast<uint2 *>(orow + f) = pk;
                }
            }
        }
    }
}

template <int D>
hipError_t launch_attention_d(const AttnArgs &a, hipStream_t stream)
{
    static LdsLimit seen;
    const void *fn = reinterpret_cast<const void *>(&sparse_attention_kernel<D>);
    hipError_t e = raise_lds_limit(fn, AttnShape<D>::LDS, seen);
    if (e != hipSuccess) return e;
    const int64_t grid = (int64_t)a.n_heads * a.n_chunks * a.tiles_per_chunk;
    hipLaunchKernelGGL((sparse_attention_kernel<D>), dim3((unsigned)grid), dim3(kAT), AttnShape<D>::LDS, stream, a);
    return hipGetLastError();
}

}  // namespace

bool attention_supported(int dtype, int d) { return dtype == 1 && (d == 64 || d == 128); }

int attention_tiles_per_chunk(int chunk) { return (chunk + kQT - 1) / kQT; }

hipError_t launch_attention(const AttnArgs &a, hipStream_t stream)
{
    if (a.d == 128) return launch_attention_d<128>(a, stream);
    return launch_attention_d<64>(a, stream);
}

hipError_t launch_pool(const void *X, int n_heads, int n_tok, int d, int chunk, int dtype, void *out,
                       hipStream_t stream)
{
    const int nc = (n_tok + chunk - 1) / chunk;
    const int vec = dtype == 1 ? 8 : 4;
    const int tl = kPoolThreads / (d / vec);
    const size_t lds = (size_t)tl * d * sizeof(float);
    const dim3 grid((unsigned)((int64_t)n_heads * nc));
    if (dtype == 1)
        hipLaunchKernelGGL(pool_kernel<bf16_t>, grid, dim3(kPoolThreads), lds, stream,
                           static_cast<const bf16_t *>(X), n_tok, d, chunk, nc, static_cast<bf16_t *>(out));
    else
        hipLaunchKernelGGL(pool_kernel<float>, grid, dim3(kPoolThreads), lds, stream, static_cast<const float *>(X),
                           n_tok, d, chunk, nc, static_cast<float *>(out));
    return hipGetLastError();
}

hipError_t launch_expand(const int32_t *routes, int64_t rows, int k, int chunk, int n_tok, int32_t *tokens,
                         hipStream_t stream)
{
    const int64_t total = rows * k * (int64_t)chunk;
    const int64_t want = (total + 255) / 256;
    const unsigned grid = (unsigned)(want < 65536 ? (want > 0 ? want : 1) : 65536);
    hipLaunchKernelGGL(expand_kernel, dim3(grid), dim3(256), 0, stream, routes, rows, k, chunk, n_tok, tokens);
    return hipGetLastError();
}

}  // namespace rr
