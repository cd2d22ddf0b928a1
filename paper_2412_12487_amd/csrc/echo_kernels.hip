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
#include "echo_internal.h"

namespace echo {
namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;  // SplitMix64 increment
constexpr uint64_t kMixA = 0xBF58476D1CE4E5B9ull;    // SplitMix64 output function
constexpr uint64_t kMixB = 0x94D049BB133111EBull;
constexpr int64_t kKnobLimit = int64_t(1) << 40;
constexpr int64_t kInf = INT64_MAX;

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

__global__ __launch_bounds__(64) void k_walk(WalkArgs a) {
    const int lane = threadIdx.x;
    const int32_t r = blockIdx.x / a.tiles;
    const int32_t tile = a.tile0 + blockIdx.x % a.tiles;
    const int32_t sig0 = tile * kLanes + lane;
    const bool active = sig0 < a.n_scen;
    const int32_t sigma = active ? sig0 : a.n_scen - 1;   // idle lanes mirror the last scenario
    const int64_t ns = a.n_scen;
    const echo_scenario *sc = a.scen + sigma;
    const uint64_t jseed = sc->jitter_seed;
    const uint32_t jstream = sc->jitter_stream;
    const int32_t amp = sc->jitter_amp_q16;
    const bool use_factor = a.factor != nullptr;
    const bool final_pass = a.final_pass != 0;
    const bool want_digest = final_pass && a.digest != nullptr;
    const unsigned *tile_count = a.count + tile;

    // Per stream: finish of the latest op, or a comm op still waiting for its barrier.
    int64_t lf[kStreams], ps[kStreams];
    int32_t pc[kStreams], pv[kStreams];
#pragma unroll
    for (int j = 0; j < kStreams; ++j) {
        lf[j] = 0;
        ps[j] = 0;
        pc[j] = -1;
        pv[j] = 0;
    }
    int64_t smax = 0;
    uint64_t dig = 0;
    unsigned err = 0;
    const int64_t beg = a.rank_off[r], end = a.rank_off[r + 1];
    const int4 *items4 = reinterpret_cast<const int4 *>(a.items);
    int4 nlo = make_int4(0, 0, 0, 0), nhi = nlo;
    if (beg + lane < end) {
        nlo = items4[2 * (beg + lane)];
        nhi = items4[2 * (beg + lane) + 1];
    }

// Finish of the comm op pending on stream j: barrier (latest member launch) + cost.
#define RESOLVE(j)                                                                               \
    if (pc[j] >= 0) {                                                                            \
        const int64_t c_ = pc[j];                                                                \
        if (!wait_arrivals(tile_count + c_ * a.n_tiles, (unsigned)a.c_N[c_], a.status,           \
                           a.spin_limit))                                                        \
            goto out;                                                                            \
        const uint64_t b_ = __hip_atomic_fetch_max(a.arrive + c_ * ns + sigma, 0ull,             \
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  \
        const int64_t f_ = (int64_t)b_ + a.cost[c_ * ns + sigma];                                \
        err |= f_ >= kTimeLimit ? kStatusOverflow : 0u;                                          \
        if (active) a.finish[(int64_t)pv[j] * ns + sigma] = f_;                                  \
        if (final_pass) {                                                                        \
            smax = f_ > smax ? f_ : smax;                                                        \
            if (want_digest) dig += mix64(mix64((uint64_t)pv[j] ^ (uint64_t)ps[j]) ^ (uint64_t)f_); \
        }                                                                                        \
        lf[j] = f_;                                                                              \
        pc[j] = -1;                                                                              \
    }

    for (int64_t blk = beg; blk < end; blk += kLanes) {
        // lane j holds item blk + j; the next block is fetched while this one runs
        const int4 clo = nlo, chi = nhi;
        if (blk + kLanes + lane < end) {
            nlo = items4[2 * (blk + kLanes + lane)];
            nhi = items4[2 * (blk + kLanes + lane) + 1];
        }
        const int nb = end - blk < kLanes ? int(end - blk) : kLanes;
        for (int j = 0; j < nb; ++j) {
            const int32_t op = __builtin_amdgcn_readlane(clo.x, j);
            const uint32_t meta = (uint32_t)__builtin_amdgcn_readlane(clo.y, j);
            const int32_t nfar = __builtin_amdgcn_readlane(clo.z, j);
            const int32_t far_off = __builtin_amdgcn_readlane(clo.w, j);
            const int32_t coll = __builtin_amdgcn_readlane(chi.x, j);
            const int64_t dur = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(chi.w, j) << 32) |
                                          (uint32_t)__builtin_amdgcn_readlane(chi.z, j));
            const int kind = item_kind(meta), st = item_stream(meta);
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
                const int64_t fu = a.finish[u * ns + sigma];
                ready = fu > ready ? fu : ready;
            }
            const int64_t row = (int64_t)op * ns + sigma;
            if (kind == ECHO_COMM) {
                // launch: publish this member's launch time, then count the arrival
                if (active) {
                    a.start[row] = ready;
                    __hip_atomic_fetch_max(a.arrive + (int64_t)coll * ns + sigma,
                                           (unsigned long long)ready, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                }
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
                if (use_factor && kind == ECHO_COMPUTE) d = q16(d, a.factor[row]);
                const int64_t f = ready + d;
                err |= f >= kTimeLimit ? kStatusOverflow : 0u;
                if (active) {
                    a.start[row] = ready;
                    a.finish[row] = f;
                }
#pragma unroll
                for (int q = 0; q < kStreams; ++q)
                    if (q == st) lf[q] = f;
                if (final_pass) {
                    smax = f > smax ? f : smax;
                    if (want_digest) dig += mix64(mix64((uint64_t)op ^ (uint64_t)ready) ^ (uint64_t)f);
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < kStreams; ++q) { RESOLVE(q) }
#undef RESOLVE
out:
    if (active) {
        if (err) __hip_atomic_fetch_or(a.status, err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (final_pass) {
            __hip_atomic_fetch_max(reinterpret_cast<unsigned long long *>(a.step) + sigma,
                                   (unsigned long long)smax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (want_digest)
                __hip_atomic_fetch_add(reinterpret_cast<unsigned long long *>(a.digest) + sigma,
                                       (unsigned long long)dig, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ------------------------------------------------------------------ overlap detection
// One wavefront per (rank, tile).  Compute ops of one stream run back to back,
// and so do the comm ops of one stream, so for each comm stream a cursor that
// only moves forward finds every comm op overlapping the current compute op.
__global__ __launch_bounds__(64) void k_overlap(OverlapArgs a) {
    const int lane = threadIdx.x;
    const int32_t r = blockIdx.x / a.n_tiles;
    const int32_t tile = blockIdx.x % a.n_tiles;
    const int32_t sig0 = tile * kLanes + lane;
    const bool active = sig0 < a.n_scen;
    const int32_t sigma = active ? sig0 : a.n_scen - 1;
    const int64_t ns = a.n_scen;
    const uint32_t *slow = &a.scen[sigma].slowdown_q16[0][0];
    const int64_t *cl_off = a.cl_off + (int64_t)r * kStreams;
    const int64_t *cp_off = a.cp_off + (int64_t)r * kStreams;

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
            if (cl_off[k + 1] > cl_off[k]) {
                const int64_t c = a.cl[cl_off[k]];
                cs[k] = a.start[c * ns + sigma];
                cf[k] = a.finish[c * ns + sigma];
            }
        }
        for (int64_t i = b0; i < b1; ++i) {
            const int64_t v = a.cp[i];
            const int cls = a.cp_class[i];
            const int64_t sv = a.start[v * ns + sigma], fv = a.finish[v * ns + sigma];
            uint32_t F = 65536u;
#pragma unroll
            for (int k = 0; k < kStreams; ++k) {
                const int64_t kb = cl_off[k];
                const int32_t nk = (int32_t)(cl_off[k + 1] - kb);
                if (nk == 0) continue;
                while (cf[k] <= sv) {                  // ends before v starts: never again
                    ++p[k];
                    if (p[k] < nk) {
                        const int64_t c = a.cl[kb + p[k]];
                        cs[k] = a.start[c * ns + sigma];
                        cf[k] = a.finish[c * ns + sigma];
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
                        const uint32_t x = slow[cls * kTypes + a.cl_type[kb + q]];
                        F = x > F ? x : F;
                    }
                    if (qf >= fv) break;               // the next one starts after v ends
                    if (++q >= nk) break;
                    const int64_t c = a.cl[kb + q];
                    qs = a.start[c * ns + sigma];
                    qf = a.finish[c * ns + sigma];
                }
            }
            if (active) a.factor[v * ns + sigma] = F;
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
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k_walk),
                                      dim3((unsigned)(n_ranks * a.tiles)), dim3(kLanes), params, 0, stream);
}

hipError_t launch_overlap(const OverlapArgs &a, int32_t n_ranks, hipStream_t stream) {
    hipLaunchKernelGGL(k_overlap, dim3((unsigned)(n_ranks * a.n_tiles)), dim3(kLanes), 0, stream, a);
    return hipGetLastError();
}

hipError_t walk_capacity(int device, int64_t *waves) {
    int per_cu = 0, cus = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(k_walk),
                                                                kLanes, 0);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    *waves = (int64_t)per_cu * cus;
    return hipSuccess;
}

}  // namespace echo
