// echo_kernels.hip -- gfx950 kernels of the timeline composer.
//
//   k_init     clear barrier state and outputs, check scenario ranges
//   k_clear    clear barrier state between passes
//   k_cc_cost  CC estimator (Sec. 5.3, Eq. 2-5): one lane per (collective, scenario)
//   k_walk     timeline composer (Sec. 4.2) with the collective synchronisation
//              rule (Sec. 5.2): one wavefront per (rank, 64-scenario tile) walks
//              the rank's ops in level order, max-plus relaxation in registers
//   k_overlap  validator input (Sec. 6): per compute op and scenario, the largest
//              slowdown factor over the comm ops of its rank that overlap it
//
// Everything is int64 nanoseconds and Q16 factors, bit-exact by construction:
// max, add, 64-bit multiply and shifts only (no floating point on the path).
#include <algorithm>

#include "echo_internal.h"

namespace echo {
namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;  // SplitMix64 increment
constexpr uint64_t kMixA = 0xBF58476D1CE4E5B9ull;    // SplitMix64 output function
constexpr uint64_t kMixB = 0x94D049BB133111EBull;
constexpr int64_t kKnobLimit = int64_t(1) << 40;
constexpr int64_t kInf = INT64_MAX;
// s_waitcnt immediate for "vmcnt(0)" on gfx9-family targets (expcnt and lgkmcnt left at their maxima)
constexpr int kWaitVm0 = 0x0F70;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * kMixA;
    z = (z ^ (z >> 27)) * kMixB;
    return z ^ (z >> 31);
}

// (d * f + 2^15) >> 16 in unsigned 64-bit: d < 2^44 and f < 2^20 never wrap.
__device__ __forceinline__ int64_t q16(int64_t d, uint64_t f) {
    return int64_t(((uint64_t)d * f + 32768ull) >> 16);
}

// Base duration with uniform jitter of amplitude amp (Q16) from the
// (jstream * 2^36 + v + 1)-th SplitMix64 output of the scenario's seed.
__device__ __forceinline__ int64_t jittered(int64_t d0, int32_t v, uint64_t seed, uint32_t jstream,
                                            int32_t amp) {
    const uint64_t k = ((uint64_t)jstream << 36) + (uint64_t)(uint32_t)v + 1ull;
    const uint64_t u = mix64(seed + k * kGolden);
    const int64_t J = (int64_t)(((u >> 32) * (uint64_t)(2 * amp + 1)) >> 32) - amp;
    return q16(d0, (uint64_t)(65536 + J));
}

__device__ __forceinline__ int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

__device__ __forceinline__ int64_t clog2(int64_t x) {
    int64_t k = 0;
    while ((int64_t(1) << k) < x) ++k;
    return k;
}

__device__ __forceinline__ unsigned ld_relaxed(const unsigned *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ set-up
__global__ void k_init(const echo_scenario *scen, int32_t n_scen, unsigned long long *arrive,
                       int64_t n_arrive, unsigned *count, int64_t n_count, int64_t *step,
                       uint64_t *digest, unsigned *status) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = tid; i < n_arrive; i += nth) arrive[i] = 0;
    for (int64_t i = tid; i < n_count; i += nth) count[i] = 0;
    for (int64_t i = tid; i < n_scen; i += nth) {
        if (step) step[i] = 0;
        if (digest) digest[i] = 0;
        const echo_scenario &s = scen[i];
        bool ok = s.alpha_ns >= 0 && s.alpha_ns < kKnobLimit && s.bw_intra_MBps >= 1 &&
                  s.bw_intra_MBps < kKnobLimit && s.bw_inter_MBps >= 1 &&
                  s.bw_inter_MBps < kKnobLimit && s.reduce_MBps >= 1 &&
                  s.reduce_MBps < kKnobLimit && s.jitter_amp_q16 >= 0 &&
                  s.jitter_amp_q16 <= 65535 && s.ar_algo <= ECHO_TREE;
        for (int k = 0; k < kClasses; ++k)
            for (int t = 0; t < kTypes; ++t) {
                const uint32_t f = s.slowdown_q16[k][t];
                ok = ok && f >= 65536u && f < (1u << 20);
            }
        if (!ok) __hip_atomic_fetch_or(status, kStatusRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

__global__ void k_clear(unsigned long long *arrive, int64_t n_arrive, unsigned *count, int64_t n_count) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = tid; i < n_arrive; i += nth) arrive[i] = 0;
    for (int64_t i = tid; i < n_count; i += nth) count[i] = 0;
}

// ------------------------------------------------------------------ CC estimator
// One block per collective; lanes stride over scenarios.
__global__ __launch_bounds__(64) void k_cc_cost(DeviceGraph g, const echo_scenario *scen,
                                                int32_t n_scen, int64_t *cost) {
    const int64_t c = blockIdx.x;
    const int type = g.c_type[c];
    const int64_t S = g.c_bytes[c], chunk = g.c_chunk[c];
    const int64_t N = g.c_N[c], M = g.c_M[c], K = g.c_K[c];
    const unsigned __int128 eta_ring = (unsigned __int128)g.c_eta_ring[c];
    const unsigned __int128 eta_chunks = (unsigned __int128)g.c_eta_chunks[c];
    const unsigned __int128 n1 = (unsigned __int128)(N - 1);
    for (int32_t s = threadIdx.x; s < n_scen; s += blockDim.x) {
        const echo_scenario &sc = scen[s];
        // invalid knobs are reported by k_init; keep the divisions defined
        const int64_t bwa = sc.bw_intra_MBps >= 1 ? sc.bw_intra_MBps : 1;
        const int64_t bwe = sc.bw_inter_MBps >= 1 ? sc.bw_inter_MBps : 1;
        const int64_t red = sc.reduce_MBps >= 1 ? sc.reduce_MBps : 1;
        const unsigned __int128 alpha = (unsigned __int128)(sc.alpha_ns >= 0 ? sc.alpha_ns : 0);
        const unsigned __int128 beta = (unsigned __int128)cdiv(chunk * 1000, bwa);
        const unsigned __int128 gamma = (unsigned __int128)cdiv(chunk * 1000, bwe);
        const unsigned __int128 hop = M > 1 ? gamma : beta;
        const unsigned __int128 reduce = (unsigned __int128)cdiv(S * 1000, red);
        unsigned __int128 T;
        if (type == ECHO_AG) {
            T = alpha + hop * eta_ring * n1;                                    // Eq. 2
        } else if (type == ECHO_RS) {
            T = alpha + eta_ring * (n1 * beta + n1 * hop) + reduce;             // Eq. 3
        } else if (type == ECHO_AR) {
            if (sc.ar_algo == ECHO_TREE)                                        // Eq. 5
                T = alpha + hop * (eta_chunks > 0 ? eta_chunks - 1 : 0) +
                    2 * beta * (unsigned __int128)(K - 1) +
                    2 * hop * (unsigned __int128)clog2(M) + reduce;
            else                                                                // Eq. 4
                T = alpha + eta_ring * (n1 * beta + 2 * n1 * hop) + reduce;
        } else {                                                                // P2P
            T = alpha + eta_chunks * hop;
        }
        if (T >= (unsigned __int128)kTimeLimit) {
            __hip_atomic_fetch_or(g.status, kStatusOverflow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            T = (unsigned __int128)(kTimeLimit - 1);
        }
        cost[c * n_scen + s] = (int64_t)T;
    }
}

// ------------------------------------------------------------------ composer
// Wait until `need` member wavefronts of one scenario tile have published
// their launch times.  Bounded: gives up (and tells every other waiter to give
// up) after spin_limit ticks of the 100 MHz wall clock.
__device__ bool wait_arrivals(const unsigned *cnt, unsigned need, unsigned *status, int64_t limit) {
    if (__builtin_amdgcn_readfirstlane(ld_relaxed(cnt)) >= need) return true;
    const uint64_t t0 = wall_clock64();
    for (;;) {
        __builtin_amdgcn_s_sleep(2);
        if (__builtin_amdgcn_readfirstlane(ld_relaxed(cnt)) >= need) return true;
        if (__builtin_amdgcn_readfirstlane(ld_relaxed(status)) & kStatusAbort) return false;
        if ((int64_t)(wall_clock64() - t0) > limit) {
            __hip_atomic_fetch_or(status, kStatusTimeout | kStatusAbort, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
    }
}

constexpr int kBlock = 32;   // walk items fetched (and factors staged) per round

// One wavefront walks one rank's list for one 64-scenario tile.  REFINED: the
// pass inflates compute ops by the factors of the previous pass's overlaps.
// FINAL: the pass produces the step time (and DIGEST: the timeline digest).
template <bool REFINED, bool FINAL, bool DIGEST>
__global__ __launch_bounds__(64) void k_walk(WalkArgs a) {
    __shared__ uint32_t fstage[REFINED ? kBlock * kLanes : 1];
    const int lane = threadIdx.x;
    const int32_t r = blockIdx.x / a.tiles;
    const int32_t tile = a.tile0 + blockIdx.x % a.tiles;
    const int32_t sig0 = tile * kLanes + lane;
    const bool active = sig0 < a.n_scen;
    // Idle lanes of the last tile mirror its last scenario: they compute the same
    // values and store them to the same places; only active lanes issue atomics.
    const int32_t col = active ? lane : a.n_scen - 1 - tile * kLanes;
    const bool mirror = (tile + 1) * kLanes > a.n_scen;
    const int32_t sigma = tile * kLanes + col;
    const int64_t ns = a.n_scen;
    const echo_scenario *sc = a.scen + sigma;
    const uint64_t jseed = sc->jitter_seed;
    const uint32_t jstream = sc->jitter_stream;
    const int32_t amp = sc->jitter_amp_q16;
    int64_t *const sbase = a.start + (int64_t)tile * kLanes;    // row v of tile: sbase + v * ns
    int64_t *const fbase = a.finish + (int64_t)tile * kLanes;
    const unsigned *tile_count = a.count + tile;

    // Per slot: finish of the latest op, or a comm op still waiting for its barrier.
    int64_t lf[kStreams], ps[kStreams];
    int32_t pc[kStreams], pv[kStreams];
#pragma unroll
    for (int j = 0; j < kStreams; ++j) {
        lf[j] = 0;
        ps[j] = 0;
        pc[j] = -1;
        pv[j] = 0;
    }
    uint64_t dig = 0;
    uint32_t hi_or = 0;          // OR of the high words of every time: bit 30 set <=> some time >= 2^62
    unsigned err = 0;
    const int64_t beg = a.rank_off[r], end = a.rank_off[r + 1];
    // lane j < 32 holds the first half of item j of the round, lane 32 + j its second half
    const int4 *items4 = reinterpret_cast<const int4 *>(a.items);
    const int half = lane >> 5, slotl = lane & 31;
    // lanes past the end of the list hold op 0, so staged factor loads stay in bounds
    int4 nxt = beg + slotl < end ? items4[2 * (beg + slotl) + half] : make_int4(0, 0, 0, 0);

// Finish of the comm op pending on slot j: barrier (latest member launch) + cost.
#define RESOLVE(j)                                                                               \
    if (pc[j] >= 0) {                                                                            \
        const int64_t c_ = pc[j];                                                                \
        if (!wait_arrivals(tile_count + c_ * a.n_tiles, (unsigned)a.c_N[c_], a.status,           \
                           a.spin_limit))                                                        \
            goto out;                                                                            \
        uint64_t b_ = 0;                                                                         \
        if (active)                                                                              \
            b_ = __hip_atomic_fetch_max(a.arrive + c_ * ns + sigma, 0ull, __ATOMIC_RELAXED,      \
                                        __HIP_MEMORY_SCOPE_AGENT);                               \
        b_ = mirror ? (uint64_t)__shfl((long long)b_, col) : b_;                                 \
        const int64_t f_ = (int64_t)b_ + a.cost[c_ * ns + sigma];                                \
        hi_or |= (uint32_t)((uint64_t)f_ >> 32);                                                 \
        (fbase + (int64_t)pv[j] * ns)[col] = f_;                                                 \
        if (DIGEST) dig += mix64(mix64((uint64_t)pv[j] ^ (uint64_t)ps[j]) ^ (uint64_t)f_);       \
        lf[j] = f_;                                                                              \
        pc[j] = -1;                                                                              \
    }

    for (int64_t blk = beg; blk < end; blk += kBlock) {
        const int4 cur = nxt;
        const int nb = end - blk < kBlock ? int(end - blk) : kBlock;
        nxt = blk + kBlock + slotl < end ? items4[2 * (blk + kBlock + slotl) + half] : make_int4(0, 0, 0, 0);
        if (REFINED) {
            // stage this round's slowdown factors: one load per item, one wait per round
            uint32_t fv[kBlock];
#pragma unroll
            for (int j = 0; j < kBlock; ++j) {
                const int32_t opj = __builtin_amdgcn_readlane(cur.x, j);
                fv[j] = a.factor[(int64_t)opj * ns + sigma];
            }
#pragma unroll
            for (int j = 0; j < kBlock; ++j) fstage[j * kLanes + lane] = fv[j];
        }
        for (int j = 0; j < nb; ++j) {
            const int32_t op = __builtin_amdgcn_readlane(cur.x, j);
            const uint32_t meta = (uint32_t)__builtin_amdgcn_readlane(cur.y, j);
            const int64_t dur = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.y, j + 32) << 32) |
                                          (uint32_t)__builtin_amdgcn_readlane(cur.x, j + 32));
            const int kind = item_kind(meta);
            if (meta & kFast) {
                // compute/memcpy op right after the previous op of slot 0
                int64_t d = amp != 0 ? jittered(dur, op, jseed, jstream, amp) : dur;
                if (REFINED && kind == ECHO_COMPUTE) d = q16(d, fstage[j * kLanes + lane]);
                const int64_t s0 = lf[0], f = s0 + d;
                (sbase + (int64_t)op * ns)[col] = s0;
                (fbase + (int64_t)op * ns)[col] = f;
                hi_or |= (uint32_t)((uint64_t)f >> 32);
                if (DIGEST) dig += mix64(mix64((uint64_t)op ^ (uint64_t)s0) ^ (uint64_t)f);
                lf[0] = f;
                continue;
            }
            const int32_t far_off = __builtin_amdgcn_readlane(cur.z, j);
            const int32_t coll = __builtin_amdgcn_readlane(cur.w, j);
            const int32_t nfar = __builtin_amdgcn_readlane(cur.z, j + 32);
            const int st = item_stream(meta);
            const unsigned mask = item_regmask(meta);
            int64_t ready = 0;
#pragma unroll
            for (int q = 0; q < kStreams; ++q) {
                if (mask & (1u << q)) {
                    RESOLVE(q)
                    ready = lf[q] > ready ? lf[q] : ready;
                }
            }
            for (int32_t q = 0; q < nfar; ++q) {
                const int64_t u = a.far[far_off + q];
                const int64_t fu = (fbase + u * ns)[col];
                ready = fu > ready ? fu : ready;
            }
            (sbase + (int64_t)op * ns)[col] = ready;
            if (kind == ECHO_COMM) {
                // launch: publish this member's launch time, then count the arrival
                if (active)
                    __hip_atomic_fetch_max(a.arrive + (int64_t)coll * ns + sigma, (unsigned long long)ready,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                if (lane == 0)
                    __hip_atomic_fetch_add(a.count + (int64_t)coll * a.n_tiles + tile, 1u,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                for (int q = 0; q < kStreams; ++q)
                    if (q == st) {
                        pc[q] = coll;
                        pv[q] = op;
                        ps[q] = ready;
                    }
            } else {
                int64_t d = amp != 0 ? jittered(dur, op, jseed, jstream, amp) : dur;
                if (REFINED && kind == ECHO_COMPUTE) d = q16(d, fstage[j * kLanes + lane]);
                const int64_t f = ready + d;
                hi_or |= (uint32_t)((uint64_t)f >> 32);
                (fbase + (int64_t)op * ns)[col] = f;
                if (DIGEST) dig += mix64(mix64((uint64_t)op ^ (uint64_t)ready) ^ (uint64_t)f);
#pragma unroll
                for (int q = 0; q < kStreams; ++q)
                    if (q == st) lf[q] = f;
            }
        }
    }
#pragma unroll
    for (int q = 0; q < kStreams; ++q) { RESOLVE(q) }
#undef RESOLVE
    if (hi_or >> 30) err |= kStatusOverflow;
    if (active && err) __hip_atomic_fetch_or(a.status, err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (FINAL && active) {
        // finishes along a FIFO stream never decrease: the last op of each slot holds its maximum
        int64_t smax = 0;
#pragma unroll
        for (int q = 0; q < kStreams; ++q) smax = lf[q] > smax ? lf[q] : smax;
        __hip_atomic_fetch_max(reinterpret_cast<unsigned long long *>(a.step) + sigma, (unsigned long long)smax,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (DIGEST)
            __hip_atomic_fetch_add(reinterpret_cast<unsigned long long *>(a.digest) + sigma,
                                   (unsigned long long)dig, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
out:
    if (active && err) __hip_atomic_fetch_or(a.status, err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

using WalkKernel = void (*)(WalkArgs);
WalkKernel walk_kernel(bool refined, bool final_pass, bool digest) {
    if (!final_pass) return refined ? k_walk<true, false, false> : k_walk<false, false, false>;
    if (digest) return refined ? k_walk<true, true, true> : k_walk<false, true, true>;
    return refined ? k_walk<true, true, false> : k_walk<false, true, false>;
}

// ------------------------------------------------------------------ overlap detection
// One wavefront per (rank, tile).  Compute ops of one stream run back to back,
// and so do the comm ops of one stream, so for each comm stream a cursor that
// only moves forward finds every comm op overlapping the current compute op.
// After compute op v the cursor of each comm stream sits on the first comm op
// that ends after v started; for the next compute op v', "that comm op starts
// at or after v' ends" proves both "no overlap" and "cursor stays" -- one
// compare per comm stream in the common case.  A compute op's interval is
// rebuilt rather than read: a chained op starts where the previous compute op
// of its stream finished, and every finish is start + base duration (the same
// jitter draw as the composer pass, inflated by the factor that pass used);
// only unchained ops read their start.
__global__ __launch_bounds__(64) void k_overlap(OverlapArgs a) {
    const int lane = threadIdx.x;
    const int32_t r = blockIdx.x / a.n_tiles;
    const int32_t tile = blockIdx.x % a.n_tiles;
    const bool active = tile * kLanes + lane < a.n_scen;
    const int32_t col = active ? lane : a.n_scen - 1 - tile * kLanes;
    const int32_t sigma = tile * kLanes + col;
    const int64_t ns = a.n_scen;
    const int64_t *const sbase = a.start + (int64_t)tile * kLanes;
    const int64_t *const fbase = a.finish + (int64_t)tile * kLanes;
    uint32_t *const obase = a.factor + (int64_t)tile * kLanes;
    const echo_scenario *sc = a.scen + sigma;
    const uint32_t *slow = &sc->slowdown_q16[0][0];
    const uint64_t jseed = sc->jitter_seed;
    const uint32_t jstream = sc->jitter_stream;
    const int32_t amp = sc->jitter_amp_q16;
    const int64_t *cl_off = a.cl_off + (int64_t)r * kStreams;
    const int64_t *cp_off = a.cp_off + (int64_t)r * kStreams;

    // comm streams of this rank that carry comm ops, packed to the front
    int64_t kb[kStreams];
    int32_t nk[kStreams];
    int ncs = 0;
#pragma unroll
    for (int k = 0; k < kStreams; ++k) {
        kb[k] = 0;
        nk[k] = 0;
    }
    for (int k = 0; k < kStreams; ++k) {
        const int64_t b = cl_off[k], n = cl_off[k + 1] - b;
        if (n == 0) continue;
#pragma unroll
        for (int q = 0; q < kStreams; ++q)
            if (q == ncs) {
                kb[q] = b;
                nk[q] = (int32_t)n;
            }
        ++ncs;
    }

    for (int s = 0; s < kStreams; ++s) {
        const int64_t b0 = cp_off[s], b1 = cp_off[s + 1];
        if (b0 == b1) continue;
        int32_t p[kStreams];
        int64_t cs[kStreams], cf[kStreams];
#pragma unroll
        for (int k = 0; k < kStreams; ++k) {
            p[k] = 0;
            cs[k] = kInf;
            cf[k] = kInf;
            if (k < ncs) {
                const int64_t c = a.cl[kb[k]];
                cs[k] = (sbase + c * ns)[col];
                cf[k] = (fbase + c * ns)[col];
            }
        }
        int64_t fprev = 0;
        // lane j holds compute record i0 + j of the current round of 64
        const int4 *recs = reinterpret_cast<const int4 *>(a.cp);
        int4 nxt = b0 + lane < b1 ? recs[b0 + lane] : make_int4(0, 0, 0, 0);
        for (int64_t i0 = b0; i0 < b1; i0 += kLanes) {
            const int4 cur = nxt;
            // settle the round's records here, once, so the per-op loop below carries
            // no memory wait (a wait there would also wait for the previous op's store)
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
            nxt = i0 + kLanes + lane < b1 ? recs[i0 + kLanes + lane] : make_int4(0, 0, 0, 0);
            const int nr = b1 - i0 < kLanes ? int(b1 - i0) : kLanes;
            for (int j = 0; j < nr; ++j) {
                const int64_t v = __builtin_amdgcn_readlane(cur.x, j);
                const int meta = __builtin_amdgcn_readlane(cur.y, j);
                const int64_t d0 = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.w, j) << 32) |
                                             (uint32_t)__builtin_amdgcn_readlane(cur.z, j));
                const int64_t sv = (meta & kChained) ? fprev : (sbase + v * ns)[col];
                int64_t d = amp != 0 ? jittered(d0, (int32_t)v, jseed, jstream, amp) : d0;
                if (a.prev_refined) d = q16(d, (obase + v * ns)[col]);   // the previous pass's duration
                const int64_t fv = sv + d;
                fprev = fv;
                bool busy = false;
    #pragma unroll
                for (int k = 0; k < kStreams; ++k)
                    if (k < ncs) busy |= cs[k] < fv;
                uint32_t F = 65536u;
                if (busy) {
                    const int cls = meta & 7;
    #pragma unroll
                    for (int k = 0; k < kStreams; ++k) {
                        if (k >= ncs) break;
                        if (!(cs[k] < fv)) continue;
                        while (cf[k] <= sv) {              // ends before v starts: never again
                            ++p[k];
                            if (p[k] < nk[k]) {
                                const int64_t c = a.cl[kb[k] + p[k]];
                                cs[k] = (sbase + c * ns)[col];
                                cf[k] = (fbase + c * ns)[col];
                            } else {
                                cs[k] = kInf;
                                cf[k] = kInf;
                            }
                        }
                        int32_t q = p[k];
                        int64_t qs = cs[k], qf = cf[k];
                        while (qs < fv) {
                            const int64_t lo = sv > qs ? sv : qs, hi = fv < qf ? fv : qf;
                            if (lo < hi) {
                                const uint32_t x = slow[cls * kTypes + a.cl_type[kb[k] + q]];
                                F = x > F ? x : F;
                            }
                            if (qf >= fv) break;           // the next one starts after v ends
                            if (++q >= nk[k]) break;
                            const int64_t c = a.cl[kb[k] + q];
                            qs = (sbase + c * ns)[col];
                            qf = (fbase + c * ns)[col];
                        }
                    }
                }
                (obase + v * ns)[col] = F;
            }
        }
    }
}

int grid_for(int64_t n, int block) {
    int64_t b = (n + block - 1) / block;
    if (b < 1) b = 1;
    if (b > 65536) b = 65536;
    return (int)b;
}

}  // namespace

hipError_t launch_init(const DeviceGraph &g, const echo_scenario *scen, int32_t n_scen,
                       unsigned long long *arrive, int64_t n_arrive, unsigned *count, int64_t n_count,
                       int64_t *step, uint64_t *digest, hipStream_t stream) {
    int64_t n = n_arrive > n_count ? n_arrive : n_count;
    if (n_scen > n) n = n_scen;
    hipLaunchKernelGGL(k_init, dim3(grid_for(n, 256)), dim3(256), 0, stream, scen, n_scen, arrive,
                       n_arrive, count, n_count, step, digest, g.status);
    return hipGetLastError();
}

hipError_t launch_clear(unsigned long long *arrive, int64_t n_arrive, unsigned *count, int64_t n_count,
                        hipStream_t stream) {
    const int64_t n = n_arrive > n_count ? n_arrive : n_count;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_clear, dim3(grid_for(n, 256)), dim3(256), 0, stream, arrive, n_arrive, count,
                       n_count);
    return hipGetLastError();
}

hipError_t launch_cc_cost(const DeviceGraph &g, const echo_scenario *scen, int32_t n_scen, int64_t *cost,
                          hipStream_t stream) {
    if (g.n_colls == 0 || n_scen == 0) return hipSuccess;
    hipLaunchKernelGGL(k_cc_cost, dim3((unsigned)g.n_colls), dim3(64), 0, stream, g, scen, n_scen, cost);
    return hipGetLastError();
}

hipError_t launch_walk(const WalkArgs &a, int32_t n_ranks, hipStream_t stream) {
    WalkArgs args = a;
    void *params[] = {&args};
    const WalkKernel k = walk_kernel(a.factor != nullptr, a.final_pass != 0, a.digest != nullptr);
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k), dim3((unsigned)(n_ranks * a.tiles)),
                                      dim3(kLanes), params, 0, stream);
}

hipError_t launch_overlap(const OverlapArgs &a, int32_t n_ranks, hipStream_t stream) {
    hipLaunchKernelGGL(k_overlap, dim3((unsigned)(n_ranks * a.n_tiles)), dim3(kLanes), 0, stream, a);
    return hipGetLastError();
}

hipError_t walk_capacity(int device, int64_t *waves) {
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    int64_t least = INT64_MAX;
    for (int v = 0; v < 8; ++v) {
        int per_cu = 0;
        const WalkKernel k = walk_kernel(v & 1, v & 2, v & 4);
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(k), kLanes, 0);
        if (e != hipSuccess) return e;
        least = std::min<int64_t>(least, (int64_t)per_cu * cus);
    }
    *waves = least;
    return hipSuccess;
}

}  // namespace echo
