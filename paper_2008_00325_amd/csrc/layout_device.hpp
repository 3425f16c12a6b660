// layout_device.hpp -- device-side building blocks of the layout SGD for gfx950.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), the per-epoch edge
// schedule, the two gradient coefficients of the cross-entropy objective
// (UMAP section; Phi = 1/(1 + a d^(2b))), and the fixed-point accumulator
// that makes the epoch-synchronous update independent of summation order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ul {

constexpr int kWave = 64;

// Stream tags in the fourth counter word (one value per random stream).
constexpr uint32_t kTagInit = 0x494E0000u;
constexpr uint32_t kTagNeg = 0x4E470000u;

constexpr float kClip = 4.0f;      // per-component gradient clip
constexpr float kRepEps = 1e-3f;   // regulariser of d^2 in the repulsion
// Fixed-point accumulator: 2^32 units per embedding unit, int64.  Integer adds
// are associative, so the sum of a vertex's updates does not depend on the
// order in which lanes, waves or kernels add them.
constexpr double kFixOne = 4294967296.0;
constexpr double kFixUnit = 1.0 / 4294967296.0;

struct Ctr {
    uint32_t w[4];
};

// a ^ b ^ c in one v_bitop3_b32 (truth table 0x96)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Philox4x32 with 10 rounds.  Each round multiplies counter words 0 and 2 by
// the two round constants (full 64-bit products, one v_mad_u64_u32 each); the
// high halves are mixed with words 1 and 3 and the round key (one three-input
// xor each), and the key advances by the two Weyl increments.
__device__ __forceinline__ Ctr philox4x32_10(Ctr c, uint32_t key_lo, uint32_t key_hi)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.w[0];
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.w[2];
        Ctr nx;
        nx.w[0] = xor3((uint32_t)(p1 >> 32), c.w[1], key_lo);
        nx.w[1] = (uint32_t)p1;
        nx.w[2] = xor3((uint32_t)(p0 >> 32), c.w[3], key_hi);
        nx.w[3] = (uint32_t)p0;
        c = nx;
        key_lo += 0x9E3779B9u;
        key_hi += 0xBB67AE85u;
    }
    return c;
}

// Words of negative samples 4q .. 4q+3 of edge e in epoch `epoch`.
__device__ __forceinline__ Ctr negative_words(int64_t e, int32_t epoch, int32_t q, uint32_t key_lo,
                                              uint32_t key_hi)
{
    Ctr c;
    c.w[0] = (uint32_t)(uint64_t)e;
    c.w[1] = (uint32_t)((uint64_t)e >> 32);
    c.w[2] = (uint32_t)epoch;
    c.w[3] = kTagNeg | (uint32_t)q;
    return philox4x32_10(c, key_lo, key_hi);
}

// Uniform vertex in [0, n) from a 32-bit word: the high half of u * n.
__device__ __forceinline__ uint32_t word_to_vertex(uint32_t u, uint32_t n) { return __umulhi(u, n); }

// Edge e with epochs-per-sample eps is sampled in epoch `epoch` when the
// number of whole periods elapsed grows across the epoch (fp32, IEEE
// division).
__device__ __forceinline__ bool edge_active(float eps, int32_t epoch)
{
    float now = floorf((float)(epoch + 1) / eps);
    float before = floorf((float)epoch / eps);
    return now > before;
}

__device__ __forceinline__ float clip4(float g) { return fminf(fmaxf(g, -kClip), kClip); }

// d2^b for d2 > 0 by the hardware base-2 logarithm and exponential.
__device__ __forceinline__ float pow_b(float d2, float b) { return __builtin_amdgcn_exp2f(b * __builtin_amdgcn_logf(d2)); }

// Attraction: d/dy_i log Phi = c (y_i - y_j), c = -2ab d2^(b-1) / (1 + a d2^b),
// written as -2ab d2^b / (d2 (1 + a d2^b)) with one hardware reciprocal; 0
// when the points coincide.  Branch-free (the guard is a select).  Valid for
// d2 >= kTinyD2 only: below it the hardware logarithm and reciprocal, which
// take no subnormal input, would turn the product into 0 * inf
// (attraction_grad handles that range).
constexpr float kTinyD2 = 0x1p-60f;
__device__ __forceinline__ float attraction_coef(float d2, float a, float b)
{
    const float p = pow_b(d2, b);
    const float c = (-2.0f * a * b * p) * __builtin_amdgcn_rcpf(d2 * fmaf(a, p, 1.0f));
    return d2 > 0.0f ? c : 0.0f;
}

// The clipped attraction of a pair 0 < d2 < kTinyD2 (every component of the
// difference below 2^-30 in magnitude, d2 possibly subnormal or flushed to 0
// by the squares).  The difference is scaled by 2^88 (exact), so that its
// squared norm d2s lies in [2^-122, 2^121] for any nonzero fp32 difference,
// and each component is evaluated in the log domain:
//   |c diff_d| = 2ab * q * |diff_d| / d2 = 2^(log2(2ab) + log2 q + 88 + log2(|ds_d| / d2s)),
//   q = p / (1 + a p), p = d2^b, log2 q = b L - log2(1 + a 2^(b L)), L = log2(d2s) - 176,
// which neither overflows nor loses p to underflow; the sign is that of -diff_d.
// Rare by construction (coincident or nearly coincident endpoints), so the
// extra transcendentals and the IEEE division do not matter.
template <int DIM>
__device__ __forceinline__ void attraction_tiny(const float (&diff)[DIM], float a, float b, float (&g)[DIM])
{
    constexpr float kS = 0x1p88f;
    float ds[DIM];
    float d2s = 0.0f;
#pragma unroll
    for (int d = 0; d < DIM; ++d) {
        ds[d] = diff[d] * kS;
        d2s = fmaf(ds[d], ds[d], d2s);
    }
    const float bl = b * (__builtin_amdgcn_logf(d2s) - 176.0f);
    const float lq = bl - __builtin_amdgcn_logf(fmaf(a, __builtin_amdgcn_exp2f(bl), 1.0f));
    const float base = __builtin_amdgcn_logf(2.0f * a * b) + lq + 88.0f;
#pragma unroll
    for (int d = 0; d < DIM; ++d) {
        const float m = __builtin_amdgcn_exp2f(base + __builtin_amdgcn_logf(fabsf(ds[d]) / d2s));
        g[d] = d2s > 0.0f ? copysignf(fminf(m, kClip), -ds[d]) : 0.0f;
    }
}

// Clipped attraction gradient of a pair with difference `diff` (y_i - y_j)
// and squared distance d2: g_d = clip(c diff_d, -4, 4), 0 when the points
// coincide (C14 of the readings: the term of a zero distance is 0).
template <int DIM>
__device__ __forceinline__ void attraction_grad(const float (&diff)[DIM], float d2, float a, float b, float (&g)[DIM])
{
    const float c = attraction_coef(d2, a, b);
#pragma unroll
    for (int d = 0; d < DIM; ++d) g[d] = clip4(c * diff[d]);
    bool tiny = false;
#pragma unroll
    for (int d = 0; d < DIM; ++d) tiny |= diff[d] != 0.0f;
    tiny &= d2 < kTinyD2;
    if (tiny) attraction_tiny<DIM>(diff, a, b, g);
}

// Repulsion: d/dy_i log(1 - Phi) = c (y_i - y_k), c = 2b / ((1e-3 + d2)(1 + a d2^b));
// 0 when the points coincide.  Branch-free.
__device__ __forceinline__ float repulsion_coef(float d2, float a, float b)
{
    const float p = pow_b(d2, b);
    const float c = (2.0f * b) * __builtin_amdgcn_rcpf((kRepEps + d2) * fmaf(a, p, 1.0f));
    return d2 > 0.0f ? c : 0.0f;
}

struct EpochArgs {
    const float *E;      // snapshot E_n of the moving vertices, n x DIM
    float *E_next;       // E_{n+1}
    const float *T;      // table of tails and negative samples: E itself, or a frozen layout (transform)
    uint32_t n;
    uint32_t row_first;  // rows [row_first, row_last) are updated (one GPU's share of a row-sharded
    uint32_t row_last;   // layout); the wave kernels get them through their partition
    uint32_t n_table;    // rows of T; negative samples are drawn from [0, n_table)
    int32_t same_table;  // T is E: a draw equal to the source is skipped, near tails may come from LDS
    int32_t in_place;    // asynchronous: E_next is E, and every launch adds its sums to the rows it owns
    float attr_mult;     // 2 when the reverse edge's equal share lands on the row too (symmetric B), else 1
    int32_t epoch;
    int32_t neg_rate;
    float a, b;
    double alpha;        // 1 - epoch / n_epochs
    uint32_t key_lo, key_hi;
    int32_t *counts;     // this epoch's row of per-wave sampled-edge counts
};

template <int DIM>
__device__ __forceinline__ float sq_dist(const float (&x)[DIM], const float (&y)[DIM], float (&diff)[DIM])
{
    float d2 = 0.0f;
#pragma unroll
    for (int d = 0; d < DIM; ++d) {
        diff[d] = x[d] - y[d];
        d2 = fmaf(diff[d], diff[d], d2);
    }
    return d2;
}

// base[i] addressed by a 32-bit byte offset (i * sizeof(T) < 2^32): a
// uniform base pointer plus one 32-bit register, the SGPR-base form of the
// global loads and stores.
template <typename T>
__device__ __forceinline__ T &at32(T *base, uint32_t i)
{
    return *reinterpret_cast<T *>(reinterpret_cast<char *>(base) + (uint32_t)(i * (uint32_t)sizeof(T)));
}
template <typename T>
__device__ __forceinline__ const T &at32(const T *base, uint32_t i)
{
    return *reinterpret_cast<const T *>(reinterpret_cast<const char *>(base) + (uint32_t)(i * (uint32_t)sizeof(T)));
}

template <int DIM>
__device__ __forceinline__ void load_row(const float *__restrict__ E, uint32_t v, float (&y)[DIM])
{
#pragma unroll
    for (int d = 0; d < DIM; ++d) y[d] = E[(size_t)v * DIM + d];
}

// One update term in fixed point: round(t * 2^32) to nearest (ties to even),
// by adding the 1.5 * 2^52 shifter in fp64 (exact for |t| < 2^19) and
// reading the integer out of the mantissa.  Every term is converted on its
// own, so the integer sum of a vertex's terms does not depend on how the
// terms are grouped into kernels, lanes or waves.
__device__ __forceinline__ long long to_fixed(float t)
{
    const double shifter = 0x1.8p52;
    const double y = fma((double)t, kFixOne, shifter);
    return (long long)(__double_as_longlong(y) - __double_as_longlong(shifter));
}

// Attraction share of vertex i for a sampled edge (i -> j): `mult` times the
// clipped gradient of log Phi.  In a fit mult = 2: the row's own "move the
// source" share plus the equal share of the reverse edge (j -> i), which is
// sampled in the same epochs because B is symmetric with bit-equal weights.
// In a transform (j frozen, no reverse edge) mult = 1.
template <int DIM>
__device__ __forceinline__ void attraction_fixed(const float (&yi)[DIM], const float (&yj)[DIM], float a, float b,
                                                 float mult, long long (&fx)[DIM])
{
    float diff[DIM], g[DIM];
    const float d2 = sq_dist<DIM>(yi, yj, diff);
    attraction_grad<DIM>(diff, d2, a, b, g);
#pragma unroll
    for (int d = 0; d < DIM; ++d) fx[d] = to_fixed(mult * g[d]);
}

// Repulsion of vertex i from a negative sample k (callers skip k == i).
template <int DIM>
__device__ __forceinline__ void repulsion_fixed(const float (&yi)[DIM], const float (&yk)[DIM], float a, float b,
                                                long long (&fx)[DIM])
{
    float diff[DIM];
    const float d2 = sq_dist<DIM>(yi, yk, diff);
    const float c = repulsion_coef(d2, a, b);
#pragma unroll
    for (int d = 0; d < DIM; ++d) fx[d] = to_fixed(clip4(c * diff[d]));
}

// The random words of negative samples 0 .. 4*NQ-1 of edge e; NQ > 0 draws
// them all at once (neg_rate <= 4 NQ).
template <int NQ>
__device__ __forceinline__ void negative_words_all(int64_t e, int32_t epoch, uint32_t key_lo, uint32_t key_hi,
                                                   uint32_t (&u)[4 * NQ])
{
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        Ctr w = negative_words(e, epoch, q, key_lo, key_hi);
#pragma unroll
        for (int t = 0; t < 4; ++t) u[4 * q + t] = w.w[t];
    }
}

// E_{n+1}[i][d] = E_n[i][d] + alpha * (accumulated fixed-point sum).
__device__ __forceinline__ float commit(float y, long long acc, double alpha)
{
    return (float)((double)y + alpha * ((double)acc * kFixUnit));
}

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wavefronts per workgroup of the edge-parallel kernels.
constexpr int kWavesPerBlock = 4;
// Rows staged in LDS on each side of a wave's own rows (by the kernels that
// stage a halo): the attraction reads y_j from there when j is that close
// (neighbour lists of locally ordered vertices), and from global memory
// otherwise.
constexpr int kHalo = 64;

__device__ __forceinline__ int64_t uniform64(int64_t v)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Logical wave index of this lane's wave in a grid of a multiple of 8
// workgroups.  Workgroups are dispatched round-robin over the 8 XCDs; each XCD
// gets a contiguous run of logical blocks so that neighbouring rows (and their
// mostly-local neighbours) share one L2.
__device__ __forceinline__ int64_t logical_wave()
{
    const int64_t per_xcd = gridDim.x / 8;
    const int64_t lb = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    return lb * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

__device__ __forceinline__ unsigned lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Number of set bits of `mask` below the calling lane.
__device__ __forceinline__ unsigned lanes_below(unsigned long long mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

}  // namespace ul
