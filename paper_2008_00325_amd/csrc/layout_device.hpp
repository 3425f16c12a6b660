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

// Philox4x32 with 10 rounds.  Each round multiplies counter words 0 and 2 by
// the two round constants; the high halves are mixed with words 1 and 3 and
// the round key, and the key advances by the two Weyl increments.
__device__ __forceinline__ Ctr philox4x32_10(Ctr c, uint32_t key_lo, uint32_t key_hi)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint32_t m0 = 0xD2511F53u, m1 = 0xCD9E8D57u;
        uint32_t hi0 = __umulhi(m0, c.w[0]);
        uint32_t lo0 = m0 * c.w[0];
        uint32_t hi1 = __umulhi(m1, c.w[2]);
        uint32_t lo1 = m1 * c.w[2];
        Ctr nx;
        nx.w[0] = hi1 ^ c.w[1] ^ key_lo;
        nx.w[1] = lo1;
        nx.w[2] = hi0 ^ c.w[3] ^ key_hi;
        nx.w[3] = lo0;
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

// Attraction: d/dy_i log Phi = c (y_i - y_j), c = -2ab d2^(b-1) / (1 + a d2^b).
__device__ __forceinline__ float attraction_coef(float d2, float a, float b)
{
    if (!(d2 > 0.0f)) return 0.0f;
    float p = exp2f(b * log2f(d2));   // d2^b
    return -2.0f * a * b * p / (d2 * (1.0f + a * p));
}

// Repulsion: d/dy_i log(1 - Phi) = c (y_i - y_k), c = 2b / ((1e-3 + d2)(1 + a d2^b)).
__device__ __forceinline__ float repulsion_coef(float d2, float a, float b)
{
    if (!(d2 > 0.0f)) return 0.0f;
    float p = exp2f(b * log2f(d2));
    return 2.0f * b / ((kRepEps + d2) * (1.0f + a * p));
}

struct EpochArgs {
    const float *E;      // snapshot E_n, n x DIM
    float *E_next;       // E_{n+1}
    uint32_t n;
    int32_t epoch;
    int32_t neg_rate;
    float a, b;
    double alpha;        // 1 - epoch / n_epochs
    uint32_t key_lo, key_hi;
    unsigned long long *active_count;  // += sampled edges of this epoch
};

// Everything one sampled edge e = (i -> j) contributes to vertex i, in
// fixed point: twice the clipped attraction (its own "move the source" share
// plus the equal share of the reverse edge (j -> i), which is sampled in the
// same epochs because B is symmetric with bit-equal weights), then the clipped
// repulsions of its negative samples (a draw equal to i is skipped).  The step
// size is applied once per vertex at the end of the epoch.
template <int DIM>
__device__ __forceinline__ void edge_contribution(const EpochArgs &A, int64_t e, uint32_t i, uint32_t j,
                                                  const float (&yi)[DIM], long long (&fx)[DIM])
{
    const float *__restrict__ E = A.E;
    float diff[DIM];
    float d2 = 0.0f;
#pragma unroll
    for (int d = 0; d < DIM; ++d) {
        diff[d] = yi[d] - E[(size_t)j * DIM + d];
        d2 += diff[d] * diff[d];
    }
    double s[DIM];
    float c = attraction_coef(d2, A.a, A.b);
#pragma unroll
    for (int d = 0; d < DIM; ++d) s[d] = 2.0 * (double)clip4(c * diff[d]);

    for (int32_t q = 0; q * 4 < A.neg_rate; ++q) {
        Ctr w = negative_words(e, A.epoch, q, A.key_lo, A.key_hi);
#pragma unroll
        for (int32_t t = 0; t < 4; ++t) {
            if (4 * q + t >= A.neg_rate) break;
            uint32_t k = word_to_vertex(w.w[t], A.n);
            if (k == i) continue;
            float dk[DIM];
            float q2 = 0.0f;
#pragma unroll
            for (int d = 0; d < DIM; ++d) {
                dk[d] = yi[d] - E[(size_t)k * DIM + d];
                q2 += dk[d] * dk[d];
            }
            float cr = repulsion_coef(q2, A.a, A.b);
#pragma unroll
            for (int d = 0; d < DIM; ++d) s[d] += (double)clip4(cr * dk[d]);
        }
    }
#pragma unroll
    for (int d = 0; d < DIM; ++d) fx[d] = __double2ll_rn(s[d] * kFixOne);
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

__device__ __forceinline__ unsigned lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Number of set bits of `mask` below the calling lane.
__device__ __forceinline__ unsigned lanes_below(unsigned long long mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

}  // namespace ul
