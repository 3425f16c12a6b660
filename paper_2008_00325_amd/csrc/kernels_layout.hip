// kernels_layout.hip -- random initialisation and the epoch kernels of the
// layout SGD (UMAP section objective; embedding-updates section), gfx950.
//
// Both epoch paths implement one epoch-synchronous step: every read sees the
// snapshot E_n, every term is converted to fixed point on its own and summed in
// int64, and E_{n+1} = E_n + alpha * sum is written to the other buffer (no
// scatter to global memory, no atomics on the embedding in global memory).
// In a transform the tails and negative samples are rows of a frozen layout T
// (the trained embedding) and only the new points, the rows of E, move.
//  * edge-parallel (default): one k_epoch_draw launch and, when the vertex
//    table is split into P > 1 ranges, P k_epoch_repulse launches per epoch,
//    each wavefront owning a range of whole rows (see the section comment
//    below).
//  * k_epoch_rowwise: one thread per vertex walking its row (a plain second
//    implementation used to cross-check the first).
// Because the sums are exact integers, both paths give the same bits.
#include "internal.hpp"

namespace ul {

// ---------------------------------------------------------------------------
// Initial layout: uniform on [-10, 10) from the init stream.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init(float *__restrict__ E, int64_t total, int32_t dim, uint32_t key_lo,
                                              uint32_t key_hi)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        int64_t i = t / dim;
        int32_t d = (int32_t)(t - i * dim);
        Ctr c;
        c.w[0] = (uint32_t)(uint64_t)i;
        c.w[1] = (uint32_t)((uint64_t)i >> 32);
        c.w[2] = (uint32_t)(d >> 2);
        c.w[3] = kTagInit;
        Ctr w = philox4x32_10(c, key_lo, key_hi);
        int sel = d & 3;
        uint32_t u = sel == 0 ? w.w[0] : sel == 1 ? w.w[1] : sel == 2 ? w.w[2] : w.w[3];
        // top 24 bits -> exact value in [-1, 1), then one fp32 rounding
        float unit = (float)((int32_t)(u >> 8) - (1 << 23)) * 0x1p-23f;
        E[t] = unit * 10.0f;
    }
}

hipError_t launch_init(float *E, int64_t n, int32_t dim, uint64_t seed, hipStream_t s)
{
    int64_t total = n * dim;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_init, dim3((unsigned)blocks), dim3(256), 0, s, E, total, dim, (uint32_t)seed,
                       (uint32_t)(seed >> 32));
    return hipGetLastError();
}

// Transform: each new point starts at the mean of its kept neighbours in the
// frozen layout T weighted by 1/eps_e (the edge weight over w_max), summed in
// fp64 in edge order; a point without kept edges starts at the origin.
__global__ __launch_bounds__(256) void k_init_transform(const int64_t *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col,
                                                        const float *__restrict__ eps, const float *__restrict__ T,
                                                        int64_t n, int32_t dim, float *__restrict__ E)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
        double den = 0.0;
        for (int64_t e = e0; e < e1; ++e) den += 1.0 / (double)eps[e];
        for (int32_t d = 0; d < dim; ++d) {
            double num = 0.0;
            for (int64_t e = e0; e < e1; ++e) num += (1.0 / (double)eps[e]) * (double)T[(size_t)col[e] * dim + d];
            E[(size_t)i * dim + d] = den > 0.0 ? (float)(num / den) : 0.0f;
        }
    }
}

hipError_t launch_init_transform(const int64_t *row_ptr, const int32_t *col, const float *eps, const float *T,
                                 int64_t n, int32_t dim, float *E, hipStream_t s)
{
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_init_transform, dim3((unsigned)blocks), dim3(256), 0, s, row_ptr, col, eps, T, n, dim, E);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One thread per vertex: the whole epoch for its row, term by term.
// ---------------------------------------------------------------------------
template <int DIM, int NQ>
__global__ __launch_bounds__(256) void k_epoch_rowwise(EpochArgs A, const int64_t *__restrict__ row_ptr,
                                                       const int32_t *__restrict__ col,
                                                       const float *__restrict__ eps)
{
    const uint32_t i = A.row_first + blockIdx.x * 256u + threadIdx.x;
    unsigned long long cnt = 0;
    if (i < A.row_last) {
        float yi[DIM];
        load_row<DIM>(A.E, i, yi);
        long long acc[DIM];
#pragma unroll
        for (int d = 0; d < DIM; ++d) acc[d] = 0;
        const int64_t e1 = row_ptr[i + 1];
        for (int64_t e = row_ptr[i]; e < e1; ++e) {
            if (!edge_active(eps[e], A.epoch)) continue;
            ++cnt;
            float yj[DIM];
            load_row<DIM>(A.T, (uint32_t)col[e], yj);
            long long fx[DIM];
            attraction_fixed<DIM>(yi, yj, A.a, A.b, A.attr_mult, fx);
#pragma unroll
            for (int d = 0; d < DIM; ++d) acc[d] += fx[d];
            for (int32_t q = 0; 4 * q < A.neg_rate; ++q) {
                Ctr w = negative_words(e, A.epoch, q, A.key_lo, A.key_hi);
                for (int t = 0; t < 4 && 4 * q + t < A.neg_rate; ++t) {
                    const uint32_t k = word_to_vertex(t == 0 ? w.w[0] : t == 1 ? w.w[1] : t == 2 ? w.w[2] : w.w[3],
                                                      A.n_table);
                    if (A.same_table && k == i) continue;
                    float yk[DIM];
                    load_row<DIM>(A.T, k, yk);
                    repulsion_fixed<DIM>(yi, yk, A.a, A.b, fx);
#pragma unroll
                    for (int d = 0; d < DIM; ++d) acc[d] += fx[d];
                }
            }
        }
#pragma unroll
        for (int d = 0; d < DIM; ++d) A.E_next[(size_t)i * DIM + d] = commit(yi[d], acc[d], A.alpha);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if ((threadIdx.x & 63) == 0) A.counts[blockIdx.x * 4 + threadIdx.x / 64] = (int32_t)cnt;
}

// ---------------------------------------------------------------------------
// Edge-parallel wavefront kernels.
//
// Each wave owns the whole rows [part[w], part[w+1]).  An epoch is one
// k_epoch_draw launch followed by P k_epoch_repulse launches:
//  * k_epoch_draw streams eps (and col, and each edge's row inside the wave)
//    over the wave's edges, classifies every edge for this epoch and appends
//    the sampled ones -- compacted with a ballot -- to an LDS ring.  It takes
//    the ring 64 edges at a time: each lane adds its edge's attraction to the
//    wave's LDS accumulator (y_j from the wave's staged rows when j is one
//    of them or, at 1-2 components, within 64 rows of them),
//    draws the edge's negative samples and files each one as a 4-byte record
//    under the range of the vertex table it falls in.  The accumulator goes
//    to delta.  With a table of one range (P = 1) the draw kernel's FUSED
//    instance gathers each negative's row itself, adds its repulsion to the
//    accumulator and commits E_{n+1}: no records and no range launch.
//  * k_epoch_repulse (range p) reads the wave's records of range p and adds
//    their repulsions.  All gathers of one launch hit one 1/P slice of the
//    vertex table, which is sized to stay resident in an XCD's L2.  The last
//    range commits the wave's rows of E_{n+1} with coalesced stores.
// ---------------------------------------------------------------------------
// The eps / col / head stream is read in super-chunks of kSuper x 64 edges,
// three deep in registers: super-chunks s+1 and s+2 are in flight while s is
// classified (the queue only ever holds classified edges, so the depth costs
// registers, not LDS).
constexpr int kSuper = 2;
// Records per lane per step of the repulsion kernel: all of a step's gathers
// are in flight at once; fewer for wide rows, so that the two DIM-vectors per
// record stay in registers at an occupancy of several waves per SIMD.
template <int DIM>
constexpr int rep_unroll() { return DIM <= 2 ? 16 : DIM <= 4 ? 8 : DIM <= 8 ? 4 : 2; }
// LDS ring of sampled edges waiting for their attraction and draws: (tail,
// (row in wave) << 24 | edge offset in wave); holds the < 64 left over plus
// one super-chunk.
constexpr int kQueue = 256;
static_assert(kQueue >= kWave - 1 + kSuper * kWave, "queue too small");
// Halo rows staged on each side of a draw wave: only for 1-2 components.
// From 3 components on a wave owns fewer rows (86 at 3, 17 at 16) while the
// halo's LDS grows with the row width, so the halo cost more occupancy than
// its LDS reads of y_j saved (200 epochs of the 1M window graph, draw kernel
// with / without: 102.9 / 108.8 us at 2 components, 122.1 / 121.1 at 3,
// 136.8 / 132.6 at 4, 233.7 / 198.1 at 8, 733.6 / 468.6 at 16).  Without a
// halo every tail outside the wave's own rows is read from global memory.
template <int DIM>
constexpr int draw_halo() { return DIM <= 2 ? kHalo : 0; }
// LDS row stride (in elements) of a wave's int64 sums and fp32 rows.  With an
// even width of 4 or more components a row is a multiple of 16 bank words, so
// lanes holding different rows of their wave meet on the same banks; one pad
// element makes the stride odd and spreads the rows over all banks.
template <int DIM>
constexpr int lds_stride() { return DIM >= 4 && DIM % 2 == 0 ? DIM + 1 : DIM; }
// LDS index of element t of a wave's rows stored back to back (t >= 0)
template <int DIM, int S>
__device__ __forceinline__ int lds_at(int t) { if constexpr (S == DIM) return t; else return (t / DIM) * S + t % DIM; }

// first vertex of table range p of P = 2^lg (ranges split the 32-bit draw)
__device__ __forceinline__ uint32_t range_base(uint32_t p, int32_t lg, uint32_t n)
{
    return lg == 0 ? 0u : __umulhi(p << (32 - lg), n);
}

// FIT: the tails and negatives index the moving layout itself (a fit: near
// tails from LDS, self draws skipped, both shares of the attraction); else they
// index a frozen table (a transform).  C16: the tails are read as 16-bit
// offsets from their rows (G.col16), 2 bytes per edge instead of 4.  FUSED:
// the table is one range (G.n_phases == 1) and each negative's repulsion is
// applied here; a separate instance, so that the record-filing kernel of
// several ranges carries none of its registers (at 8 components the draw
// launch took 222 instead of 186 us with both paths in one kernel).
template <int DIM, int NQ, bool FIT, bool C16, bool FUSED>
__global__ __launch_bounds__(256) void k_epoch_draw(EpochArgs A, WaveGraph G)
{
    constexpr int CAP = rows_cap(DIM);
    constexpr int S = lds_stride<DIM>();
    __shared__ long long s_acc[kWavesPerBlock][CAP * S];
    // a transform's tails index the frozen table: no halo
    constexpr int kHaloW = FIT ? draw_halo<DIM>() : 0;
    __shared__ float s_y[kWavesPerBlock][(CAP + 2 * kHaloW) * S];   // the wave's rows of E_n and halos
    __shared__ uint32_t s_rec[kWavesPerBlock][kMaxPhases];
    __shared__ uint2 s_q[kWavesPerBlock][kQueue];

    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const unsigned lane = threadIdx.x % kWave;
    const int64_t w = logical_wave();
    if (w >= G.n_waves) return;
    const int64_t r0 = __builtin_amdgcn_readfirstlane(G.part[w]);
    const int nrows = __builtin_amdgcn_readfirstlane(G.part[w + 1]) - (int)r0;
    if (nrows <= 0) {
        if (lane == 0) A.counts[w] = 0;
        if ((int)lane < G.n_phases) G.rec_count[(int64_t)lane * G.n_waves + w] = 0;
        return;
    }
    const int64_t e0 = uniform64(G.row_ptr[r0]);
    const int64_t e1 = uniform64(G.row_ptr[r0 + nrows]);

    long long *acc = s_acc[wv];
    float *yrows = s_y[wv] + kHaloW * S;   // row h of the wave at yrows[h * S], h in [-kHaloW, nrows + kHaloW)
    uint32_t *rec_n = s_rec[wv];
    const size_t g0 = (size_t)r0 * DIM;
    // staged rows [lo, hi): the wave's own rows and up to kHaloW on each side
    constexpr int64_t halo = kHaloW;
    const int64_t lo = r0 >= halo ? r0 - halo : 0;
    const int64_t hi = r0 + nrows + halo <= (int64_t)A.n ? r0 + nrows + halo : (int64_t)A.n;
    for (int t = lane; t < nrows * S; t += kWave) acc[t] = 0;
    if ((int)lane < kMaxPhases) rec_n[lane] = 0;
    {
        // all of a lane's row loads are issued before the first LDS store
        constexpr int kStageD = ((CAP + 2 * kHaloW) * DIM + kWave - 1) / kWave;
        float yv[kStageD];
        const int nst = (int)(hi - lo) * DIM;
#pragma unroll
        for (int q = 0; q < kStageD; ++q) {
            const int t = q * kWave + (int)lane;
            if (t < nst) yv[q] = A.E[(int64_t)lo * DIM + t];
        }
#pragma unroll
        for (int q = 0; q < kStageD; ++q) {
            const int t = q * kWave + (int)lane;
            if (t < nst) yrows[((int)(lo - r0) + t / DIM) * S + t % DIM] = yv[q];
        }
    }

    // ---- classify and compact ----------------------------------------------
    // The wave's edges are addressed by 32-bit offsets from e0 (fewer than
    // 2^24 of them) against uniform base pointers.
    const uint32_t ne = (uint32_t)(e1 - e0);
    const float *const eps_w = G.eps + e0;
    const int32_t *const col_w = G.col + e0;
    const int16_t *const col16_w = C16 ? G.col16 + e0 : nullptr;
    const uint8_t *const head_w = G.head + e0;
    int64_t qn = 0;
    // loads are unconditional (the offset is clamped into the wave's edges and
    // the value masked) so that the next super-chunk stays in flight
    auto load_super = [&](uint32_t sbase, float (&ev)[kSuper], int32_t (&cv)[kSuper],
                          uint8_t (&hv)[kSuper]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < kSuper; ++j) {
            uint32_t o = sbase + j * kWave + lane;
            o = o < ne ? o : ne - 1;
            ev[j] = at32(eps_w, o);
            if constexpr (C16)
                cv[j] = at32(col16_w, o);   // the tail's offset from its row
            else
                cv[j] = at32(col_w, o);
            hv[j] = at32(head_w, o);
        }
    };
    const int32_t R = A.neg_rate;
    const int32_t lg = G.lg_phases;
    const int64_t roff = record_offset(w, e0, R, G.n_phases);
    int64_t cap64 = (record_offset(w + 1, e1, R, G.n_phases) - roff) / G.n_phases;   // slots per range
    if (G.cap_limit >= 0 && cap64 > G.cap_limit) cap64 = G.cap_limit;
    // a wave's record slots span less than 2^32 bytes (checked by the host)
    const uint32_t cap = (uint32_t)cap64;
    uint32_t *const rec_wave = G.rec + roff;   // this wave's slots, range p from p * cap
    // One table range: the whole table stays in L2 beside the edge stream, so
    // each negative's repulsion is applied here (no records, no range launch)
    constexpr bool fused = FUSED;
    uint2 *q = s_q[wv];
    uint32_t qhead = 0, qtail = 0;
    bool overflow = false;   // a record found its range's slots full
    auto file = [&](uint32_t u, uint32_t i, int h) __attribute__((always_inline)) {
        const uint32_t k = word_to_vertex(u, A.n_table);
        if (FIT && k == i) return;   // a draw equal to the source adds nothing
        const uint32_t p = lg == 0 ? 0u : u >> (32 - lg);
        const uint32_t slot = atomicAdd(&rec_n[p], 1u);
        if (slot < cap) at32(rec_wave, p * cap + slot) = ((uint32_t)h << 24) | (k - range_base(p, lg, A.n_table));
        else overflow = true;
    };
    // repulsions of four drawn words of a lane's edge, applied at once: all
    // four table rows are loaded before the first term is computed
    auto repel4 = [&](const uint32_t *u, int cnt, uint32_t i, int h, const float (&yi)[DIM], bool live)
                      __attribute__((always_inline)) {
        uint32_t k[4];
        float yk[4][DIM];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            k[r] = word_to_vertex(u[r], A.n_table);
            if (r < cnt) load_row<DIM>(A.T, k[r], yk[r]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (r < cnt) {
                long long fx[DIM];
                repulsion_fixed<DIM>(yi, yk[r], A.a, A.b, fx);
                if (live && !(FIT && k[r] == i)) {
#pragma unroll
                    for (int d = 0; d < DIM; ++d)
                        atomicAdd(reinterpret_cast<unsigned long long *>(&acc[h * S + d]), (unsigned long long)fx[d]);
                }
            }
        }
    };
    // attraction and negative draws of `count` queued sampled edges
    auto process = [&](int count) __attribute__((always_inline)) {
        const bool valid = (int)lane < count;
        const uint2 ent = q[(qhead + lane) & (kQueue - 1)];
        const int h = valid ? (int)(ent.y >> 24) : 0;
        const int64_t e = valid ? e0 + (ent.y & 0xFFFFFFu) : e0;
        const uint32_t tail = valid ? ent.x : (uint32_t)r0;
        const uint32_t i = (uint32_t)(r0 + h);
        float yi[DIM], yj[DIM];
#pragma unroll
        for (int d = 0; d < DIM; ++d) yi[d] = yrows[h * S + d];
        // y_j from the staged rows when j is one of them, else from the table;
        // the LDS read is unconditional (a valid row otherwise) so that the
        // two reads never merge into one generic-address load
        const bool near = FIT && (int64_t)tail >= lo && (int64_t)tail < hi;
        const int64_t jt = near ? (int64_t)tail - r0 : 0;
#pragma unroll
        for (int d = 0; d < DIM; ++d) yj[d] = yrows[jt * S + d];
        if (!near) load_row<DIM>(A.T, tail, yj);
        long long fx[DIM];
        attraction_fixed<DIM>(yi, yj, A.a, A.b, FIT ? 2.0f : 1.0f, fx);
        if (valid) {
#pragma unroll
            for (int d = 0; d < DIM; ++d)
                atomicAdd(reinterpret_cast<unsigned long long *>(&acc[h * S + d]), (unsigned long long)fx[d]);
        }
        if (fused) {
            // every lane draws (the words of a lane without an edge add nothing)
            for (int32_t qq = 0; 4 * qq < R; ++qq) {
                const Ctr wd = negative_words(e, A.epoch, qq, A.key_lo, A.key_hi);
                repel4(wd.w, R - 4 * qq, i, h, yi, valid);
            }
        } else if (valid) {
            if constexpr (NQ >= 0) {
                uint32_t u[4 * NQ > 0 ? 4 * NQ : 1];
                if constexpr (NQ > 0) negative_words_all<NQ>(e, A.epoch, A.key_lo, A.key_hi, u);
#pragma unroll
                for (int r = 0; r < 4 * NQ; ++r)
                    if (r < R) file(u[r], i, h);
            } else {
                for (int32_t qq = 0; 4 * qq < R; ++qq) {
                    Ctr wd = negative_words(e, A.epoch, qq, A.key_lo, A.key_hi);
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (4 * qq + t < R) file(wd.w[t], i, h);
                }
            }
        }
        qhead += (uint32_t)count;
    };
    auto scan_super = [&](uint32_t sbase, const float (&ev)[kSuper], const int32_t (&cv)[kSuper],
                          const uint8_t (&hv)[kSuper]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < kSuper; ++j) {
            const uint32_t o = sbase + j * kWave + lane;
            if (sbase + j * kWave >= ne) break;
            const bool act = edge_active(ev[j], A.epoch) & (o < ne);
            const unsigned long long m = __ballot(act);
            if (act) {
                const uint32_t tail = C16 ? (uint32_t)((int32_t)r0 + (int32_t)hv[j] + cv[j]) : (uint32_t)cv[j];
                q[(qtail + lanes_below(m)) & (kQueue - 1)] = make_uint2(tail, ((uint32_t)hv[j] << 24) | o);
            }
            const uint32_t nact = (uint32_t)__popcll(m);
            qn += nact;
            qtail += nact;
        }
        if (qtail - qhead >= (uint32_t)kWave) {
            wave_sync();
            do {
                process(kWave);
            } while (qtail - qhead >= (uint32_t)kWave);
        }
    };
    if (ne > 0) {
        float ea[kSuper], eb[kSuper], ec[kSuper];
        int32_t ca[kSuper], cb[kSuper], cc[kSuper];
        uint8_t ha[kSuper], hb[kSuper], hc[kSuper];
        constexpr uint32_t kStep = (uint32_t)kSuper * kWave;
        load_super(0, ea, ca, ha);
        load_super(kStep, eb, cb, hb);
        for (uint32_t s0 = 0; s0 < ne; s0 += 3 * kStep) {
            load_super(s0 + 2 * kStep, ec, cc, hc);
            scan_super(s0, ea, ca, ha);
            if (s0 + kStep >= ne) break;
            load_super(s0 + 3 * kStep, ea, ca, ha);
            scan_super(s0 + kStep, eb, cb, hb);
            if (s0 + 2 * kStep >= ne) break;
            load_super(s0 + 4 * kStep, eb, cb, hb);
            scan_super(s0 + 2 * kStep, ec, cc, hc);
        }
    }
    if (qtail != qhead) {
        wave_sync();
        process((int)(qtail - qhead));
    }
    wave_sync();

    if (A.in_place || fused) {
        for (int t = lane; t < nrows * DIM; t += kWave)
            A.E_next[g0 + t] = commit(yrows[lds_at<DIM, S>(t)], acc[lds_at<DIM, S>(t)], A.alpha);
    } else {
        for (int t = lane; t < nrows * DIM; t += kWave) G.delta[g0 + t] = acc[lds_at<DIM, S>(t)];
    }
    if ((int)lane < G.n_phases) G.rec_count[(int64_t)lane * G.n_waves + w] = (int32_t)rec_n[lane];
    // per-wave count, summed by a separate pass (a global atomic per wave on
    // one address would serialise thousands of waves)
    if (lane == 0) A.counts[w] = (int32_t)qn;
    if (__ballot(overflow) != 0 && lane == 0) atomicOr(G.overflow, 1u);
}

// Waves per SIMD the repulsion kernel's registers are held to: at 1-2
// components 96 instead of 98 registers give a fifth wave per SIMD (window
// graphs: 50.6 -> 50.3 us per launch at 1M vertices, 183.8 -> 180.6 us at 5M),
// at 16 components 76 instead of 109 (1M vertices: 191.0 -> 185.7 us); other
// widths keep the compiler's choice (at 15 components the cap measured 230.3
// against 228.1 us, at 8 components 125.0 against 124.2).
template <int DIM>
constexpr int rep_waves() { return DIM <= 2 || DIM == 16 ? 5 : 1; }

template <int DIM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(rep_waves<DIM>(), 8))) void k_epoch_repulse(
    EpochArgs A, WaveGraph G, int32_t phase)
{
    constexpr int CAP = rows_cap(DIM);
    constexpr int S = lds_stride<DIM>();
    __shared__ long long s_acc[kWavesPerBlock][CAP * S];
    __shared__ float s_y[kWavesPerBlock][CAP * S];   // the wave's own rows of E_n

    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const unsigned lane = threadIdx.x % kWave;
    const int64_t w = logical_wave();
    if (w >= G.n_waves) return;
    const int64_t r0 = __builtin_amdgcn_readfirstlane(G.part[w]);
    const int nrows = __builtin_amdgcn_readfirstlane(G.part[w + 1]) - (int)r0;
    if (nrows <= 0) return;
    const int64_t e0 = uniform64(G.row_ptr[r0]);
    const int64_t e1 = uniform64(G.row_ptr[r0 + nrows]);
    const int64_t roff = record_offset(w, e0, A.neg_rate, G.n_phases);
    int64_t cap = (record_offset(w + 1, e1, A.neg_rate, G.n_phases) - roff) / G.n_phases;
    if (G.cap_limit >= 0 && cap > G.cap_limit) cap = G.cap_limit;
    int64_t nrec = __builtin_amdgcn_readfirstlane(G.rec_count[(int64_t)phase * G.n_waves + w]);
    nrec = nrec < cap ? nrec : cap;
    const bool last = phase + 1 == G.n_phases;

    long long *acc = s_acc[wv];
    float *yrows = s_y[wv];
    const size_t g0 = (size_t)r0 * DIM;
    const uint32_t *recs = G.rec + roff + (int64_t)phase * cap;
    const uint32_t base = range_base((uint32_t)phase, G.lg_phases, A.n_table);
    // kRepUnroll records per lane per step, all loads issued before use.  The
    // first step's record loads and gathers are issued around the loads of the
    // wave's rows and sums, so that those latencies overlap.
    constexpr int kRepUnroll = rep_unroll<DIM>();
    uint32_t r[kRepUnroll];
    float yk[kRepUnroll][DIM];
    if (nrec > 0) {
#pragma unroll
        for (int u = 0; u < kRepUnroll; ++u) {
            const int64_t t = u * kWave + lane;
            r[u] = recs[t < nrec ? t : 0];
        }
    }
    constexpr int kStage = (CAP * DIM + kWave - 1) / kWave;   // a wave holds at most CAP rows
    long long dv[kStage];
    float yv[kStage];
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
        const int t = q * kWave + (int)lane;
        if (t < nrows * DIM) {
            dv[q] = A.in_place ? 0ll : G.delta[g0 + t];
            yv[q] = A.E[g0 + t];
        }
    }
    if (nrec > 0) {
#pragma unroll
        for (int u = 0; u < kRepUnroll; ++u) load_row<DIM>(A.T, base + (r[u] & 0xFFFFFFu), yk[u]);
    }
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
        const int t = q * kWave + (int)lane;
        if (t < nrows * DIM) {
            acc[lds_at<DIM, S>(t)] = dv[q];
            yrows[lds_at<DIM, S>(t)] = yv[q];
        }
    }
    wave_sync();

    for (int64_t b = 0; b < nrec; b += kRepUnroll * kWave) {
        if (b > 0) {
#pragma unroll
            for (int u = 0; u < kRepUnroll; ++u) {
                const int64_t t = b + u * kWave + lane;
                r[u] = recs[t < nrec ? t : 0];
            }
#pragma unroll
            for (int u = 0; u < kRepUnroll; ++u) load_row<DIM>(A.T, base + (r[u] & 0xFFFFFFu), yk[u]);
        }
        float yi[kRepUnroll][DIM];
#pragma unroll
        for (int u = 0; u < kRepUnroll; ++u) {
            const int h = (int)(r[u] >> 24);
#pragma unroll
            for (int d = 0; d < DIM; ++d) yi[u][d] = yrows[h * S + d];
        }
#pragma unroll
        for (int u = 0; u < kRepUnroll; ++u) {
            long long fx[DIM];
            repulsion_fixed<DIM>(yi[u], yk[u], A.a, A.b, fx);
            const int h = (int)(r[u] >> 24);
            if (b + u * kWave + lane < nrec) {
#pragma unroll
                for (int d = 0; d < DIM; ++d)
                    atomicAdd(reinterpret_cast<unsigned long long *>(&acc[h * S + d]), (unsigned long long)fx[d]);
            }
        }
    }
    wave_sync();

    if (last || A.in_place) {
        for (int t = lane; t < nrows * DIM; t += kWave)
            A.E_next[g0 + t] = commit(yrows[lds_at<DIM, S>(t)], acc[lds_at<DIM, S>(t)], A.alpha);
    } else {
        for (int t = lane; t < nrows * DIM; t += kWave) G.delta[g0 + t] = acc[lds_at<DIM, S>(t)];
    }
}

int32_t phase_log2(int64_t n, int32_t dim)
{
    const int64_t bytes = n * dim * (int64_t)sizeof(float);
    if (bytes <= (dim <= 8 ? kOneRangeBytes : dim <= kOneRangeMaxDim ? kOneRangeBytesWide : 0)) return 0;
    int32_t lg_bytes = 0;   // the fewest ranges that bring a range down to kPhaseTableBytes
    while ((1 << (lg_bytes + 1)) <= kMaxPhases && (bytes >> lg_bytes) > kPhaseTableBytes) ++lg_bytes;
    int32_t lg_rows = 2;    // 4 ranges up to kPhaseRows vertices, twice as many per doubling of n beyond
    while ((1 << (lg_rows + 1)) <= kMaxPhases && (n >> (lg_rows - 2)) > kPhaseRows) ++lg_rows;
    return lg_bytes < lg_rows ? lg_bytes : lg_rows;
}

template <int DIM, int NQ, bool FIT, bool C16>
static void launch_draw(int64_t grid, const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    if (G.n_phases == 1)
        hipLaunchKernelGGL((k_epoch_draw<DIM, NQ, FIT, C16, true>), dim3((unsigned)grid), dim3(256), 0, s, A, G);
    else
        hipLaunchKernelGGL((k_epoch_draw<DIM, NQ, FIT, C16, false>), dim3((unsigned)grid), dim3(256), 0, s, A, G);
}

template <int DIM, int NQ>
static hipError_t launch_epoch_dq(int kernel, const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    if (kernel == 1) {
        const int64_t blocks = ((int64_t)A.row_last - A.row_first + 255) / 256;
        hipLaunchKernelGGL((k_epoch_rowwise<DIM, NQ>), dim3((unsigned)blocks), dim3(256), 0, s, A, G.row_ptr, G.col,
                           G.eps);
        return hipGetLastError();
    }
    const int64_t blocks = (G.n_waves + kWavesPerBlock - 1) / kWavesPerBlock;
    const int64_t grid = ((blocks + 7) / 8) * 8;
    // the 16-bit tail stream is compiled for the common widths (1-4 components)
    if constexpr (DIM <= 4) {
        if (A.same_table && G.col16) {
            launch_draw<DIM, NQ, true, true>(grid, A, G, s);
            for (int32_t p = 0; G.n_phases > 1 && p < G.n_phases; ++p)
                hipLaunchKernelGGL((k_epoch_repulse<DIM>), dim3((unsigned)grid), dim3(256), 0, s, A, G, p);
            return hipGetLastError();
        }
    }
    if (A.same_table)
        launch_draw<DIM, NQ, true, false>(grid, A, G, s);
    else
        launch_draw<DIM, NQ, false, false>(grid, A, G, s);
    for (int32_t p = 0; G.n_phases > 1 && p < G.n_phases; ++p)
        hipLaunchKernelGGL((k_epoch_repulse<DIM>), dim3((unsigned)grid), dim3(256), 0, s, A, G, p);
    return hipGetLastError();
}

template <int DIM>
static hipError_t launch_epoch_dim(int kernel, const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    if (A.neg_rate == 0) return launch_epoch_dq<DIM, 0>(kernel, A, G, s);
    if (A.neg_rate <= 4) return launch_epoch_dq<DIM, 1>(kernel, A, G, s);
    if (A.neg_rate <= 8) return launch_epoch_dq<DIM, 2>(kernel, A, G, s);
    return launch_epoch_dq<DIM, -1>(kernel, A, G, s);
}

hipError_t launch_epoch(int kernel, int32_t dim, const EpochArgs &A, const WaveGraph &G, hipStream_t s)
{
    switch (dim) {
#define UL_CASE(D) \
    case D: return launch_epoch_dim<D>(kernel, A, G, s);
        UL_CASE(1) UL_CASE(2) UL_CASE(3) UL_CASE(4) UL_CASE(5) UL_CASE(6) UL_CASE(7) UL_CASE(8)
        UL_CASE(9) UL_CASE(10) UL_CASE(11) UL_CASE(12) UL_CASE(13) UL_CASE(14) UL_CASE(15) UL_CASE(16)
#undef UL_CASE
    default: return hipErrorInvalidValue;
    }
}

// ---------------------------------------------------------------------------
// Sum of the per-wave counts of `rows` epochs: one block per epoch.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_reduce_counts(const int32_t *__restrict__ counts, int64_t stride,
                                                       int64_t slots, unsigned long long *__restrict__ out)
{
    const int32_t *row = counts + (int64_t)blockIdx.x * stride;
    unsigned long long s = 0;
    for (int64_t t = threadIdx.x; t < slots; t += 256) s += (unsigned long long)row[t];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    __shared__ unsigned long long s_w[4];
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = s_w[0] + s_w[1] + s_w[2] + s_w[3];
}

hipError_t launch_reduce_counts(const int32_t *counts, int64_t stride, int64_t slots, int32_t rows,
                                unsigned long long *out, hipStream_t s)
{
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_reduce_counts, dim3((unsigned)rows), dim3(256), 0, s, counts, stride, slots, out);
    return hipGetLastError();
}

// *out = a[0] + ... + a[n - 1] (one block; the per-epoch sampled-edge counts of a call)
__global__ __launch_bounds__(256) void k_sum_u64(const unsigned long long *__restrict__ a, int64_t n,
                                                 unsigned long long *__restrict__ out)
{
    unsigned long long s = 0;
    for (int64_t t = threadIdx.x; t < n; t += 256) s += a[t];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    __shared__ unsigned long long s_w[4];
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) *out = s_w[0] + s_w[1] + s_w[2] + s_w[3];
}

hipError_t launch_sum_u64(const unsigned long long *a, int64_t n, unsigned long long *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_sum_u64, dim3(1), dim3(256), 0, s, a, n, out);
    return hipGetLastError();
}

int64_t count_slots(int kernel, int64_t n, int64_t n_waves)
{
    return kernel == 1 ? ((n + 255) / 256) * 4 : n_waves;
}

// ---------------------------------------------------------------------------
// Diagnostics: the schedule and the negative draws, by the same routines.
// ---------------------------------------------------------------------------
__global__ void k_debug_active(const float *__restrict__ eps, int64_t nnz, int32_t epoch, uint8_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nnz; e += stride)
        out[e] = edge_active(eps[e], epoch) ? 1 : 0;
}

hipError_t launch_debug_active(const float *eps, int64_t nnz, int32_t epoch, uint8_t *out, hipStream_t s)
{
    int64_t blocks = (nnz + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_debug_active, dim3((unsigned)blocks), dim3(256), 0, s, eps, nnz, epoch, out);
    return hipGetLastError();
}

__global__ void k_debug_negatives(uint32_t n, uint32_t key_lo, uint32_t key_hi, int32_t epoch, int64_t e_first,
                                  int64_t count, int32_t neg_rate, uint32_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) {
        const int64_t e = e_first + t;
        for (int32_t q = 0; q * 4 < neg_rate; ++q) {
            Ctr w = negative_words(e, epoch, q, key_lo, key_hi);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (4 * q + tt >= neg_rate) break;
                out[t * neg_rate + 4 * q + tt] = word_to_vertex(w.w[tt], n);
            }
        }
    }
}

hipError_t launch_debug_negatives(uint32_t n, uint64_t seed, int32_t epoch, int64_t e_first, int64_t count,
                                  int32_t neg_rate, uint32_t *out, hipStream_t s)
{
    int64_t blocks = (count + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_debug_negatives, dim3((unsigned)blocks), dim3(256), 0, s, n, (uint32_t)seed,
                       (uint32_t)(seed >> 32), epoch, e_first, count, neg_rate, out);
    return hipGetLastError();
}

}  // namespace ul
