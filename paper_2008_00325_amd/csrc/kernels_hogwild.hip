// kernels_hogwild.hip -- the asynchronous (Hogwild) epoch of the layout SGD
// (embedding-updates and reproducibility sections): the embedding is updated
// in place while the epoch runs, each sampled edge moving both of its
// endpoints and its source again for every negative sample, with no barrier
// between the edges of an epoch.  Results depend on the timing of the
// wavefronts; the epoch-synchronous kernels are the deterministic mode.
//
// One launch per epoch, over the same wavefront partition as the
// epoch-synchronous kernels (each wave owns the whole rows [part[w],
// part[w+1])):
//  * the wave stages its rows and kHalo rows on each side in LDS, streams eps /
//    col / row-in-wave over its edges and compacts the sampled ones into an LDS
//    ring, then takes them 64 at a time, one per lane;
//  * a lane reads y_i (the staged row plus the wave's own pending updates of
//    it) and y_j (LDS when j is staged, global memory otherwise), applies the
//    attraction to a private copy of y_i and then each negative sample's
//    repulsion in turn (y_k read from the live table), so that later terms see
//    the earlier ones, as a sequential pass over the edge would;
//  * the source's change and, when j is one of the wave's rows, the
//    destination's change go to fp32 accumulators in LDS (pre-aggregation per
//    row, the local cache of the embedding-updates section); a destination
//    outside the wave's rows takes a global fp32 atomic add at once;
//  * at the end the wave adds its rows' accumulated changes to the table with
//    global atomic adds (other waves may be moving the same rows as
//    destinations).
#include "internal.hpp"

namespace ul {

namespace {

// LDS ring of sampled edges: (tail, (row in wave) << 24 | edge offset in wave);
// holds the < 64 left over plus one chunk of 64.
constexpr int kHwQueue = 128;

template <int DIM, int NQ>
__global__ __launch_bounds__(256) void k_epoch_hogwild(EpochArgs A, WaveGraph G)
{
    constexpr int CAP = rows_cap(DIM);
    __shared__ float s_y[kWavesPerBlock][(CAP + 2 * kHalo) * DIM];   // rows staged at the wave's start
    __shared__ float s_acc[kWavesPerBlock][CAP * DIM];               // pending changes of the wave's rows
    __shared__ uint2 s_q[kWavesPerBlock][kHwQueue];

    float *const E = A.E_next;   // the table, updated in place
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const unsigned lane = threadIdx.x % kWave;
    const int64_t w = logical_wave();
    if (w >= G.n_waves) return;
    const int64_t r0 = __builtin_amdgcn_readfirstlane(G.part[w]);
    const int nrows = __builtin_amdgcn_readfirstlane(G.part[w + 1]) - (int)r0;
    if (nrows <= 0) {
        if (lane == 0) A.counts[w] = 0;
        return;
    }
    const int64_t e0 = uniform64(G.row_ptr[r0]);
    const int64_t e1 = uniform64(G.row_ptr[r0 + nrows]);

    float *acc = s_acc[wv];
    float *yrows = s_y[wv] + kHalo * DIM;   // row h of the wave at yrows[h * DIM], h in [-kHalo, nrows + kHalo)
    const size_t g0 = (size_t)r0 * DIM;
    const int64_t lo = r0 >= kHalo ? r0 - kHalo : 0;
    const int64_t hi = r0 + nrows + kHalo <= (int64_t)A.n ? r0 + nrows + kHalo : (int64_t)A.n;
    for (int t = lane; t < nrows * DIM; t += kWave) acc[t] = 0.0f;
    for (int64_t t = (lo - r0) * DIM + lane; t < (hi - r0) * DIM; t += kWave) yrows[t] = E[(int64_t)g0 + t];
    wave_sync();

    const float alpha = (float)A.alpha;
    const int32_t R = A.neg_rate;
    uint2 *q = s_q[wv];
    uint32_t qhead = 0, qtail = 0;
    int64_t qn = 0;

    auto process = [&](int count) __attribute__((always_inline)) {
        const bool valid = (int)lane < count;
        const uint2 ent = q[(qhead + lane) & (kHwQueue - 1)];
        const int h = valid ? (int)(ent.y >> 24) : 0;
        const int64_t e = valid ? e0 + (ent.y & 0xFFFFFFu) : e0;
        const uint32_t tail = valid ? ent.x : (uint32_t)r0;
        const uint32_t i = (uint32_t)(r0 + h);
        const int64_t jt = (int64_t)tail - r0;   // tail's row relative to the wave
        const bool j_own = jt >= 0 && jt < nrows;

        float yi[DIM], yj[DIM];
#pragma unroll
        for (int d = 0; d < DIM; ++d) yi[d] = yrows[h * DIM + d] + acc[h * DIM + d];
        // staged copy (plus pending changes for the wave's own rows) when j is
        // staged, else the table; the LDS reads are unconditional (a valid row
        // otherwise) so that they never merge with the global read
        const bool near = (int64_t)tail >= lo && (int64_t)tail < hi;
        const int64_t jn = near ? jt : 0;
        const int64_t ja = j_own ? jt : 0;
#pragma unroll
        for (int d = 0; d < DIM; ++d) yj[d] = yrows[jn * DIM + d] + (j_own ? acc[ja * DIM + d] : 0.0f);
        if (!near) load_row<DIM>(E, tail, yj);

        // negative samples: every y_k is loaded before the sequential updates
        constexpr int kNeg = NQ > 0 ? 4 * NQ : 1;
        uint32_t kv[kNeg];
        float yk[kNeg][DIM];
        if constexpr (NQ > 0) {
            uint32_t u[4 * NQ];
            negative_words_all<NQ>(e, A.epoch, A.key_lo, A.key_hi, u);
#pragma unroll
            for (int r = 0; r < kNeg; ++r) {
                kv[r] = word_to_vertex(u[r], A.n);
                if (r < R) load_row<DIM>(E, kv[r], yk[r]);
            }
        }

        float diff[DIM], g[DIM], cur[DIM];
        const float d2 = sq_dist<DIM>(yi, yj, diff);
        attraction_grad<DIM>(diff, d2, A.a, A.b, g);
#pragma unroll
        for (int d = 0; d < DIM; ++d) cur[d] = fmaf(alpha, g[d], yi[d]);
        auto repel = [&](const float (&y)[DIM]) __attribute__((always_inline)) {
            float df[DIM];
            const float dd = sq_dist<DIM>(cur, y, df);
            const float cr = repulsion_coef(dd, A.a, A.b);
#pragma unroll
            for (int d = 0; d < DIM; ++d) cur[d] = fmaf(alpha, clip4(cr * df[d]), cur[d]);
        };
        if constexpr (NQ > 0) {
#pragma unroll
            for (int r = 0; r < kNeg; ++r)
                if (r < R && kv[r] != i) repel(yk[r]);
        } else if constexpr (NQ < 0) {
            for (int32_t qq = 0; 4 * qq < R; ++qq) {
                Ctr wd = negative_words(e, A.epoch, qq, A.key_lo, A.key_hi);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if (4 * qq + t >= R) break;
                    const uint32_t k = word_to_vertex(wd.w[t], A.n);
                    if (k == i) continue;
                    float y[DIM];
                    load_row<DIM>(E, k, y);
                    repel(y);
                }
            }
        }

        if (valid) {
#pragma unroll
            for (int d = 0; d < DIM; ++d) atomicAdd(&acc[h * DIM + d], cur[d] - yi[d]);
            if (j_own) {
#pragma unroll
                for (int d = 0; d < DIM; ++d) atomicAdd(&acc[jt * DIM + d], -alpha * g[d]);
            }
        }
        // the global adds come after a wave barrier, so that the compiler
        // cannot merge them with the LDS adds into one generic-address atomic
        wave_sync();
        if (valid && !j_own) {
#pragma unroll
            for (int d = 0; d < DIM; ++d) unsafeAtomicAdd(&E[(size_t)tail * DIM + d], -alpha * g[d]);
        }
        qhead += (uint32_t)count;
    };

    if (e1 > e0) {
        // one chunk of 64 edges in flight while the previous one is classified
        auto load = [&](int64_t base, float &ev, int32_t &cv, uint8_t &hv) __attribute__((always_inline)) {
            int64_t e = base + lane;
            e = e < e1 ? e : e1 - 1;
            ev = G.eps[e];
            cv = G.col[e];
            hv = G.head[e];
        };
        float ev;
        int32_t cv;
        uint8_t hv;
        load(e0, ev, cv, hv);
        for (int64_t base = e0; base < e1; base += kWave) {
            float en = 0.0f;
            int32_t cn = 0;
            uint8_t hn = 0;
            if (base + kWave < e1) load(base + kWave, en, cn, hn);
            const int64_t e = base + lane;
            const bool act = (e < e1) & edge_active(ev, A.epoch);
            const unsigned long long m = __ballot(act);
            if (act)
                q[(qtail + lanes_below(m)) & (kHwQueue - 1)] =
                    make_uint2((uint32_t)cv, ((uint32_t)hv << 24) | (uint32_t)(e - e0));
            const uint32_t nact = (uint32_t)__popcll(m);
            qn += nact;
            qtail += nact;
            if (qtail - qhead >= (uint32_t)kWave) {
                wave_sync();
                process(kWave);
                wave_sync();
            }
            ev = en;
            cv = cn;
            hv = hn;
        }
    }
    if (qtail != qhead) {
        wave_sync();
        process((int)(qtail - qhead));
    }
    wave_sync();

    for (int t = lane; t < nrows * DIM; t += kWave) unsafeAtomicAdd(&E[g0 + t], acc[t]);
    if (lane == 0) A.counts[w] = (int32_t)qn;
}

template <int DIM, int NQ>
hipError_t launch_dq(const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    const int64_t blocks = (G.n_waves + kWavesPerBlock - 1) / kWavesPerBlock;
    const int64_t grid = ((blocks + 7) / 8) * 8;
    hipLaunchKernelGGL((k_epoch_hogwild<DIM, NQ>), dim3((unsigned)grid), dim3(256), 0, s, A, G);
    return hipGetLastError();
}

template <int DIM>
hipError_t launch_dim(const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    if (A.neg_rate == 0) return launch_dq<DIM, 0>(A, G, s);
    if (A.neg_rate <= 4) return launch_dq<DIM, 1>(A, G, s);
    if (A.neg_rate <= 8) return launch_dq<DIM, 2>(A, G, s);
    return launch_dq<DIM, -1>(A, G, s);
}

}  // namespace

hipError_t launch_epoch_hogwild(int32_t dim, const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    switch (dim) {
#define UL_CASE(D) \
    case D: return launch_dim<D>(A, G, s);
        UL_CASE(1) UL_CASE(2) UL_CASE(3) UL_CASE(4) UL_CASE(5) UL_CASE(6) UL_CASE(7) UL_CASE(8)
        UL_CASE(9) UL_CASE(10) UL_CASE(11) UL_CASE(12) UL_CASE(13) UL_CASE(14) UL_CASE(15) UL_CASE(16)
#undef UL_CASE
    default: return hipErrorInvalidValue;
    }
}

}  // namespace ul
