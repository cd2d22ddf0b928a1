// echo_kernels.hip -- gfx950 kernels of the timeline composer.
//
//   k_init     clear barrier state and outputs, check scenario ranges
//   k_clear    clear barrier state between passes
//   k_cc_cost  CC estimator (Sec. 5.3, Eq. 2-5): one lane per (collective, scenario)
//   k_walk     timeline composer (Sec. 4.2) with the collective synchronisation
//              rule (Sec. 5.2): one wavefront per (walker, 64-scenario tile) walks
//              the ops of its ranks in level order, max-plus relaxation in registers
//   k_overlap  validator input (Sec. 6): per compute op and scenario, the mask of
//              collective types among the comm ops of its rank that overlap it
//
// Everything is int64 nanoseconds and Q16 factors, bit-exact by construction:
// max, add, 64-bit multiply and shifts only (no floating point on the path).
#include <algorithm>
#include <mutex>

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
// polls between reads of the abort bit and the clock: of a barrier in device memory (a
// poll is a memory round trip) and of one in LDS
constexpr unsigned kCheckPollsGlobal = 16;
constexpr unsigned kCheckPollsLocal = 256;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * kMixA;
    z = (z ^ (z >> 27)) * kMixB;
    return z ^ (z >> 31);
}

// (d * f + 2^15) >> 16 in unsigned 64-bit: d < 2^44 and f < 2^20 never wrap.
__device__ __forceinline__ int64_t q16(int64_t d, uint32_t f) {
    return int64_t(((uint64_t)d * (uint64_t)f + 32768ull) >> 16);
}

// Base duration with uniform jitter of amplitude amp (Q16) from the k-th
// SplitMix64 output of the scenario's seed, k = jstream * 2^36 + v + 1.  The
// SplitMix64 state seed + k * golden is split into a per-scenario part
// (base = seed + jstream * 2^36 * golden) and a per-op part ((v + 1) * golden,
// the same for every lane).  The factor is f = 65536 - amp + J with J the high word
// of the output scaled to [0, 2 amp]; the lane's constants 65536 - amp and 2 amp + 1
// are taken once.
struct Jitter {
    uint64_t base;
    uint32_t f0;      // 65536 - amp
    uint32_t span;    // 2 amp + 1
};
__device__ __forceinline__ Jitter make_jitter(uint64_t seed, uint32_t jstream, int32_t amp) {
    return Jitter{seed + ((uint64_t)jstream << 36) * kGolden, (uint32_t)(65536 - amp), (uint32_t)(2 * amp + 1)};
}
__device__ __forceinline__ uint32_t jitter_factor(int32_t v, const Jitter &jt) {
    // (v + 1) * golden is the same for every lane: two scalar multiplies (kept opaque so the
    // compiler does not fold them into a vector multiply-add with the lane's base)
    const uint32_t k = (uint32_t)v + 1u;
    uint32_t lo, hi;
    asm("s_mul_i32 %0, %1, %2" : "=s"(lo) : "s"(k), "s"((uint32_t)kGolden));
    asm("s_mul_hi_u32 %0, %1, %2" : "=s"(hi) : "s"(k), "s"((uint32_t)kGolden));
    hi += k * (uint32_t)(kGolden >> 32);
    const uint64_t u = mix64(jt.base + (((uint64_t)hi << 32) | lo));
    return jt.f0 + __umulhi((uint32_t)(u >> 32), jt.span);
}
// q16(d0, f) for a wave-uniform d0: below 2^32 (durations under 4.3 s) one 32 x 32-bit
// multiply-add gives the whole product.  The branch is explicit: left to itself the
// compiler evaluates the general two-multiply form for every d0.
__device__ __forceinline__ int64_t q16u(int64_t d0, uint32_t f) {
    const uint32_t dh = (uint32_t)((uint64_t)d0 >> 32);
    uint64_t p = (uint64_t)(uint32_t)d0 * f + 32768ull;
    if (__builtin_expect(__builtin_amdgcn_readfirstlane(dh) != 0, 0)) {
        uint32_t hp;
        asm volatile("v_mul_lo_u32 %0, %1, %2" : "=v"(hp) : "s"(dh), "v"(f));
        p += (uint64_t)hp << 32;
    }
    return (int64_t)(p >> 16);
}
__device__ __forceinline__ int64_t jittered(int64_t d0, int32_t v, const Jitter &jt) {
    return q16u(d0, jitter_factor(v, jt));
}
// the same for a base duration known to be below 2^32 ns
__device__ __forceinline__ int64_t jittered32(uint32_t d0, int32_t v, const Jitter &jt) {
    return (int64_t)(((uint64_t)d0 * jitter_factor(v, jt) + 32768ull) >> 16);
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
                       int64_t n_arrive, unsigned *count, int64_t n_count, int64_t *slots, int64_t n_slots,
                       int64_t *step, uint64_t *digest, int32_t n_tables, unsigned *status) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = tid; i < n_arrive; i += nth) arrive[i] = 0;
    for (int64_t i = tid; i < n_count; i += nth) count[i] = 0;
    for (int64_t i = tid; i < n_slots; i += nth) slots[i] = -1;
    for (int64_t i = tid; i < n_scen; i += nth) {
        if (step) step[i] = 0;
        if (digest) digest[i] = 0;
        const echo_scenario &s = scen[i];
        bool ok = s.alpha_ns >= 0 && s.alpha_ns < kKnobLimit && s.bw_intra_MBps >= 1 &&
                  s.bw_intra_MBps < kKnobLimit && s.bw_inter_MBps >= 1 &&
                  s.bw_inter_MBps < kKnobLimit && s.reduce_MBps >= 1 &&
                  s.reduce_MBps < kKnobLimit && s.jitter_amp_q16 >= 0 &&
                  s.jitter_amp_q16 <= 65535 && s.ar_algo <= ECHO_TREE && s.cc_model <= ECHO_CC_ALPHA_BETA &&
                  s.cc_table >= 0 && s.cc_table <= n_tables;
        for (int k = 0; k < kClasses; ++k)
            for (int t = 0; t < kTypes; ++t) {
                const uint32_t f = s.slowdown_q16[k][t];
                ok = ok && f >= 65536u && f < (1u << 20);
            }
        if (!ok) __hip_atomic_fetch_or(status, kStatusRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

__global__ void k_clear(unsigned long long *arrive, int64_t n_arrive, unsigned *count, int64_t n_count,
                        int64_t *slots, int64_t n_slots) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = tid; i < n_arrive; i += nth) arrive[i] = 0;
    for (int64_t i = tid; i < n_count; i += nth) count[i] = 0;
    for (int64_t i = tid; i < n_slots; i += nth) slots[i] = -1;
}

// ------------------------------------------------------------------ CC estimator
// One block per collective (or cost class); lanes stride over scenarios.
__global__ __launch_bounds__(64) void k_cc_cost(CollTable t, const echo_cc_table *tables, const echo_scenario *scen,
                                                int32_t n_scen, int64_t *cost, unsigned *status) {
    const int64_t c = blockIdx.x;
    const int type = t.type[c];
    const int64_t S = t.bytes[c];
    const int64_t N = t.N[c], M = t.M[c], K = t.K[c];
    const unsigned __int128 n1 = (unsigned __int128)(N - 1);
    for (int64_t s = (int64_t)blockIdx.y * blockDim.x + threadIdx.x; s < n_scen; s += (int64_t)gridDim.y * blockDim.x) {
        const echo_scenario &sc = scen[s];
        // invalid knobs are reported by k_init; keep the divisions defined
        const int64_t bwa = sc.bw_intra_MBps >= 1 ? sc.bw_intra_MBps : 1;
        const int64_t bwe = sc.bw_inter_MBps >= 1 ? sc.bw_inter_MBps : 1;
        const int64_t red = sc.reduce_MBps >= 1 ? sc.reduce_MBps : 1;
        unsigned __int128 alpha = (unsigned __int128)(sc.alpha_ns >= 0 ? sc.alpha_ns : 0);
        unsigned __int128 T;
        if (sc.cc_model == ECHO_CC_ALPHA_BETA) {
            // latency-bandwidth baseline: ring steps move ceil(S / N) bytes, tree steps all of S
            const int64_t B = M > 1 ? bwe : bwa;
            const int64_t part = cdiv(S, N);
            const unsigned __int128 tbp = (unsigned __int128)cdiv(part * 1000, B);
            const unsigned __int128 trp = (unsigned __int128)cdiv(part * 1000, red);
            if (type == ECHO_AG) {
                T = n1 * (alpha + tbp);
            } else if (type == ECHO_RS) {
                T = n1 * (alpha + tbp + trp);
            } else if (type == ECHO_AR) {
                if (sc.ar_algo == ECHO_TREE)
                    T = (unsigned __int128)clog2(N) * (2 * alpha + 2 * (unsigned __int128)cdiv(S * 1000, B) +
                                                       (unsigned __int128)cdiv(S * 1000, red));
                else
                    T = n1 * (2 * alpha + 2 * tbp + trp);
            } else {
                T = alpha + (unsigned __int128)cdiv(S * 1000, B);
            }
        } else {
            int64_t chunk, eta_r, eta_t, b, g, r;
            if (sc.cc_table > 0 && tables) {
                // profiled parameters: the first row whose size bound covers S
                const echo_cc_table &tb = tables[sc.cc_table - 1];
                int i = 0;
                while (i < ECHO_CC_ROWS - 1 && S > tb.max_bytes[i]) ++i;
                chunk = tb.chunk[i] >= 1 ? tb.chunk[i] : 1;
                eta_r = cdiv(S, N * chunk);
                eta_t = cdiv(S, chunk);
                alpha = (unsigned __int128)tb.alpha_ns[i];
                b = tb.beta_ns[i];
                g = tb.gamma_ns[i];
                r = tb.reduce_MBps[i] >= 1 ? tb.reduce_MBps[i] : 1;
            } else {
                chunk = t.chunk[c];
                eta_r = t.eta_ring[c];
                eta_t = t.eta_chunks[c];
                b = cdiv(chunk * 1000, bwa);
                g = cdiv(chunk * 1000, bwe);
                r = red;
            }
            const unsigned __int128 eta_ring = (unsigned __int128)eta_r, eta_chunks = (unsigned __int128)eta_t;
            const unsigned __int128 beta = (unsigned __int128)b;
            const unsigned __int128 hop = M > 1 ? (unsigned __int128)g : beta;
            const unsigned __int128 reduce = (unsigned __int128)cdiv(S * 1000, r);
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
        }
        if (T >= (unsigned __int128)kTimeLimit) {
            __hip_atomic_fetch_or(status, kStatusOverflow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            T = (unsigned __int128)(kTimeLimit - 1);
        }
        cost[c * n_scen + s] = (int64_t)T;
    }
}

// ------------------------------------------------------------------ composer
// Bounded waits.  A wait polls; every kCheckPollsGlobal-th poll of device memory (every
// kCheckPollsLocal-th of LDS) it also reads the abort bit and the 100 MHz wall clock, which
// it first reads at that poll (a clock read on the way into a wait would delay the first
// polls, and a wait is usually over within a few).  It gives up -- and tells every other
// waiter to give up -- once spin_limit ticks have passed since then.
struct WaitClock {
    uint64_t t0 = 0;
    bool started = false;
    // false: give up (abort seen, or the limit passed: then the abort bit is set)
    __device__ bool check(unsigned *status, int64_t limit) {
        if (__builtin_amdgcn_readfirstlane(ld_relaxed(status)) & kStatusAbort) return false;
        const uint64_t now = wall_clock64();
        if (!started) {
            started = true;
            t0 = now;
        } else if ((int64_t)(now - t0) > limit) {
            __hip_atomic_fetch_or(status, kStatusTimeout | kStatusAbort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
        return true;
    }
};

// Wait until `need` member wavefronts of one scenario tile have published
// their launch times.
__device__ bool wait_arrivals(const unsigned *cnt, unsigned need, unsigned *status, int64_t limit) {
    // Issue priority on the SIMD follows lateness: the last member to arrive is what the
    // others wait for, so it runs at raised priority until it next arrives early.
    if (__builtin_amdgcn_readfirstlane(ld_relaxed(cnt)) >= need) {
        __builtin_amdgcn_s_setprio(3);
        return true;
    }
    __builtin_amdgcn_s_setprio(0);
    WaitClock clk;
    for (unsigned it = 1;; ++it) {
        __builtin_amdgcn_s_sleep(2);
        if (__builtin_amdgcn_readfirstlane(ld_relaxed(cnt)) >= need) return true;
        if ((it & (kCheckPollsGlobal - 1)) == 0 && !clk.check(status, limit)) return false;
    }
}

// Barrier of a collective met through member slots: the latest launch time over
// its n members' slots p[m * ns] (m < n <= kSlotMembers), once every member of every
// lane's scenario has stored its launch (a slot reads -1 until then).  All slots are
// read in one memory round trip per poll.  Bounded like wait_arrivals; on giving up
// it returns 0 and clears *ok.
__device__ int64_t wait_slots(const int64_t *p, unsigned n, int64_t ns, unsigned *status, int64_t limit, bool *ok) {
    WaitClock clk;
    for (unsigned poll = 0;; ++poll) {
        int64_t v[kSlotMembers];
#pragma unroll
        for (int m = 0; m < kSlotMembers; ++m)
            v[m] = m < (int)n ? __hip_atomic_load(p + m * ns, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
        int64_t mx = 0;
        bool all = true;
#pragma unroll
        for (int m = 0; m < kSlotMembers; ++m) {
            all = all && v[m] >= 0;
            mx = v[m] > mx ? v[m] : mx;
        }
        if (!__builtin_amdgcn_readfirstlane(__ballot(!all) != 0)) {
            // every member had launched at the first look (poll 0): this wave was the last to
            // arrive and the others wait for it (issue priority as in wait_arrivals)
            if (poll == 0) __builtin_amdgcn_s_setprio(3);
            return mx;
        }
        if (poll == 0) __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_s_sleep(2);
        if (((poll + 1) & (kCheckPollsGlobal - 1)) == 0 && !clk.check(status, limit)) break;
    }
    *ok = false;
    return 0;
}

// Timeline stores stream through the caches (non-temporal): each (op, tile) row
// segment is written once per pass and read again only by the same wavefront
// (a far predecessor) or by the next kernel.
__device__ __forceinline__ void put(int64_t *p, int64_t v) { __builtin_nontemporal_store(v, p); }

// Duration d inflated by the slowdown factor of overlap mask m (Sec. 6): the
// largest entry of the op's class row over the collective types in m; an empty
// mask is factor 65536, which q16 maps to d itself.  tbl: the lane's table in
// LDS, entry e at tbl[e * 64 + lane].
__device__ __forceinline__ int64_t inflate(int64_t d, uint32_t m, const uint32_t *tbl, int cls, int lane) {
    if (m == 0) return d;
    uint32_t F = 65536u;
#pragma unroll
    for (int t = 0; t < kTypes; ++t)
        if ((m >> t) & 1u) {
            const uint32_t x = tbl[(cls * kTypes + t) * kLanes + lane];
            F = x > F ? x : F;
        }
    return q16(d, F);
}
// The same for a mask whose class row (entries t = 0..3 of the op's class) was read
// ahead: no branch, an empty mask keeps F = 65536.  Entry t takes part through an AND
// with bit t of m widened to a whole word (all ones or zero), and the largest is taken
// three at a time.
__device__ __forceinline__ int64_t inflate_row(int64_t d, uint32_t m, const uint32_t x[kTypes]) {
    static_assert(kTypes == 4, "two three-way maxima cover 65536 and four entries");
    uint32_t a[kTypes];
#pragma unroll
    for (int t = 0; t < kTypes; ++t) a[t] = x[t] & (uint32_t)__builtin_amdgcn_sbfe((int)m, t, 1);
    const uint32_t F0 = a[0] > 65536u ? a[0] : 65536u;
    const uint32_t F1 = F0 > a[1] ? F0 : a[1];
    const uint32_t F2 = a[2] > a[3] ? a[2] : a[3];
    return q16(d, F1 > F2 ? F1 : F2);
}
// s_waitcnt immediate for "lgkmcnt(0)" on gfx9-family targets (vmcnt and expcnt left at their maxima)
constexpr int kWaitLgkm0 = 0xC07F;

// Wait until `need` members have arrived at an LDS barrier slot of this block.
__device__ __forceinline__ unsigned ld_local(const unsigned *p) {
    return __builtin_amdgcn_readfirstlane(__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
}

__device__ bool wait_local(const unsigned *cnt, unsigned need, unsigned *status, int64_t limit) {
    if (ld_local(cnt) >= need) {
        __builtin_amdgcn_s_setprio(3);             // last to arrive: see wait_arrivals
        return true;
    }
    __builtin_amdgcn_s_setprio(0);
    WaitClock clk;
    for (unsigned it = 1;; ++it) {
        __builtin_amdgcn_s_sleep(1);
        if (ld_local(cnt) >= need) return true;
        if ((it & (kCheckPollsLocal - 1)) == 0 && !clk.check(status, limit)) return false;
    }
}

// A workgroup of kBlockWalkers wavefronts walks the walkers of one block for
// one 64-scenario tile; wavefront w walks walker block * kBlockWalkers + w.  REFINED:
// the pass inflates compute ops by the factors of the previous pass's
// overlaps.  FINAL: the pass produces the step time (and DIGEST: the digest).
// IN (kIn*): the pass's per-item input -- none (the first pass), overlap masks (REFINED)
// or prorated extra times (PRORATE), and whether only flagged rows are fetched.
// Every variant must fit two workgroups per CU (at most 128 registers): the loader sizes
// walkers to the fewest co-resident workgroups of any variant, so one variant over the
// limit would make the largest graphs walk more ranks per wavefront in every pass.
template <int IN, bool FINAL, bool DIGEST>
__global__ __launch_bounds__(kBlockWalkers * 64) __attribute__((amdgpu_waves_per_eu(4))) void k_walk(WalkArgs a) {
    constexpr bool REFINED = IN != kInNone;
    constexpr bool PRORATE = IN == kInExtFlags;
    constexpr bool kFlagged = IN == kInMaskFlags || IN == kInExtFlags;
    // staged per item and lane: overlap masks (one byte) or, prorating, extra times (32 bits)
    __shared__ __align__(16) uint32_t fstage[REFINED ? kBlockWalkers * kBlock * kLanes / (PRORATE ? 1 : 4) : 1];
    __shared__ unsigned long long lbar[kChannels][2][kLanes];   // per channel and slot: latest launch per lane
    __shared__ unsigned lcnt[kChannels][2];                      // per channel and slot: members arrived
    __shared__ int64_t ccost[kClassSlots][kLanes];               // staged class costs of this tile
    // slots 1..7 of every wave (slot 0 stays in a register); the prorating refined
    // pass has no LDS left for them and keeps them in registers
    constexpr bool kLdsSlots = !(REFINED && PRORATE);
    __shared__ int64_t slotmem[kLdsSlots ? kBlockWalkers * kStreams * kLanes : 1];
    __shared__ uint32_t slow[REFINED && !PRORATE ? kClasses * kTypes * kLanes : 1];   // lanes' slowdown tables
    static_assert(kBlockWalkers * 4 == kClasses * kTypes, "one 16-byte table slice per wavefront");

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform within a wavefront
    const int32_t blk = blockIdx.x / a.tiles;
    const int32_t tile = a.tile0 + blockIdx.x % a.tiles;
    const int32_t w = blk * kBlockWalkers + wave;
    const bool active = tile * kLanes + lane < a.n_scen;
    // Idle lanes of the last tile mirror its last scenario: they compute the same
    // values and store them to the same places; only active lanes issue global atomics.
    const int32_t col = active ? lane : a.n_scen - 1 - tile * kLanes;
    const bool mirror = (tile + 1) * kLanes > a.n_scen;
    const int32_t sigma = tile * kLanes + col;
    const int64_t ns = a.n_scen;

    // block set-up: clear the barrier channels, stage the block's class costs
    for (int i = threadIdx.x; i < kChannels * 2 * kLanes; i += blockDim.x) (&lbar[0][0][0])[i] = 0;
    if (threadIdx.x < kChannels * 2) (&lcnt[0][0])[threadIdx.x] = 0;
    if (wave < kClassSlots) {
        const int32_t cls = a.block_class[(int64_t)blk * kClassSlots + wave];
        ccost[wave][lane] = cls >= 0 ? a.class_cost[(int64_t)cls * ns + sigma] : 0;
    }
    if (REFINED && !PRORATE) {
        // entry e of the table for lane l at slow[e * 64 + l]: lanes hit distinct banks
        const uint4 t4 = reinterpret_cast<const uint4 *>(&a.scen[sigma].slowdown_q16[0][0])[wave];
        slow[(4 * wave + 0) * kLanes + lane] = t4.x;
        slow[(4 * wave + 1) * kLanes + lane] = t4.y;
        slow[(4 * wave + 2) * kLanes + lane] = t4.z;
        slow[(4 * wave + 3) * kLanes + lane] = t4.w;
    }
    __syncthreads();
    if (w >= a.n_walkers) return;
    // every scenario reached its fixed point in an earlier pass: nothing left to refine
    if (a.stable && __builtin_amdgcn_readfirstlane(__hip_atomic_load(a.stable, __ATOMIC_RELAXED,
                                                                      __HIP_MEMORY_SCOPE_AGENT)))
        return;

    const echo_scenario *sc = a.scen + sigma;
    const int32_t amp = sc->jitter_amp_q16;
    const Jitter jt = make_jitter(sc->jitter_seed, sc->jitter_stream, amp);
    // one branch for the whole wavefront: a lane without jitter draws the identity factor
    // (amplitude 0 gives f = 65536 and q16(d, 65536) = d)
    const bool any_jitter = __builtin_amdgcn_readfirstlane(__ballot(amp != 0) != 0);
    int64_t *const sbase = a.start + (int64_t)tile * kLanes;    // row v of tile: sbase + v * ns
    int64_t *const fbase = a.finish + (int64_t)tile * kLanes;
    const unsigned *tile_count = a.count + tile;
    uint8_t *const fst = reinterpret_cast<uint8_t *>(fstage) + (REFINED && !PRORATE ? wave * kBlock * kLanes : 0);
    uint32_t *const fst32 = fstage + (REFINED && PRORATE ? wave * kBlock * kLanes : 0);

    // Per slot: finish of the latest op (of a comm op: once its resolve item ran;
    // no item reads the slot in between).
    // (entry kStreams: where ops without a slot put their finish; never read as a slot)
    int64_t lf0 = 0;
    int64_t lf[kLdsSlots ? 1 : kStreams + 1];
    int64_t *const smem = slotmem + (kLdsSlots ? wave * kStreams * kLanes + lane : 0);
    if (kLdsSlots) {
#pragma unroll
        for (int j = 1; j < kStreams; ++j) smem[j * kLanes] = 0;
    } else {
#pragma unroll
        for (int j = 0; j <= kStreams; ++j) lf[j] = 0;
    }
    // slot q (q >= 1, wave-uniform); q == kStreams: the entry of ops without a slot
    auto slot_get = [&](int q) -> int64_t { return kLdsSlots ? smem[q * kLanes] : lf[q]; };
    auto slot_set = [&](int q, int64_t f) {
        if (kLdsSlots) {
            if (q < kStreams) smem[q * kLanes] = f;
        } else {
            lf[q] = f;
        }
    };
    // A wait that gave up (timeout or abort) marks the wave dead: it finishes its
    // list without waiting again; the times it writes are meaningless and the
    // status word already reports the failure.
    bool dead = false;
    int64_t xmax = 0;            // latest finish among ops kept out of the register slots
    uint64_t dig = 0;
    uint32_t hi_or = 0;          // OR of the high words of every time: bit 30 set <=> some time >= 2^62
    unsigned err = 0;
    const int64_t beg = a.walk_off[w], end = a.walk_off[w + 1];
    const uint32_t keep = a.store_all ? (kNeedS | kNeedF) : 0u;    // stores beyond each item's own needs
    // lane j < 32 holds the first half of item j of the round, lane 32 + j its second half
    const int4 *items4 = reinterpret_cast<const int4 *>(a.items);
    const int half = lane >> 5, slotl = lane & 31;
    // lanes past the end of the list hold op 0
    int4 nxt = beg + slotl < end ? items4[2 * (beg + slotl) + half] : make_int4(0, 0, 0, 0);

// Finish f_ of comm op v_ (collective c_, aux word x_): its barrier -- the
// latest member launch -- plus the collective's cost; written to the finish array.
#define MEET(c_, v_, x_, k_, f_, s_base_)                                                        \
    {                                                                                            \
        uint64_t b_ = 0;                                                                         \
        if ((x_) & kAuxLocal) {                                                                  \
            const int ch_ = aux_channel(x_), par_ = aux_parity(x_);                              \
            if (!dead && !__builtin_amdgcn_readfirstlane(                                        \
                             wait_local(&lcnt[ch_][par_], aux_expected(x_), a.status, a.spin_limit))) \
                dead = true;                                                                     \
            b_ = lbar[ch_][par_][lane];                                                          \
        } else if ((x_) & kAuxSlots) {                                                           \
            bool ok_ = true;                                                                     \
            if (!dead)                                                                           \
                b_ = (uint64_t)wait_slots(a.slots + (int64_t)(s_base_) * ns + sigma, aux_expected(x_), ns, \
                                          a.status, a.spin_limit, &ok_);                         \
            __builtin_amdgcn_s_waitcnt(kWaitVm0);    /* settled on this path, not at the join */ \
            if (!__builtin_amdgcn_readfirstlane(ok_)) dead = true;                               \
        } else {                                                                                 \
            if (!dead && !__builtin_amdgcn_readfirstlane(wait_arrivals(tile_count + (int64_t)(c_) * a.n_tiles, \
                                                                       (unsigned)a.c_N[c_], a.status, \
                                                                       a.spin_limit)))           \
                dead = true;                                                                     \
            if (active)                                                                          \
                b_ = __hip_atomic_fetch_max(a.arrive + (int64_t)(c_) * ns + sigma, 0ull,         \
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);         \
            __builtin_amdgcn_s_waitcnt(kWaitVm0);    /* settled on this path, not at the join */ \
            b_ = mirror ? (uint64_t)__shfl((long long)b_, col) : b_;                             \
        }                                                                                        \
        const int sl_ = aux_slot(x_);                                                            \
        /* The cost: from the workgroup's LDS slot, read first on every path; a class without  \
           a slot then reads device memory and waits for that load inside its own branch, so   \
           the common path carries no wait on vector memory (which on this target would also  \
           wait for every timeline store still in flight).  Distinct load kinds keep the two  \
           reads from merging into one flat load. */                                            \
        int64_t t_ = ccost[sl_ & (kClassSlots - 1)][lane];                                       \
        if (sl_ >= kClassSlots) {                                                                \
            t_ = __hip_atomic_load(a.class_cost + (int64_t)(k_) * ns + sigma, __ATOMIC_RELAXED,  \
                                   __HIP_MEMORY_SCOPE_AGENT);                                    \
            __builtin_amdgcn_s_waitcnt(kWaitVm0);                                                \
        }                                                                                        \
        f_ = (int64_t)b_ + t_;                                                                   \
        hi_or |= (uint32_t)((uint64_t)(f_) >> 32);                                               \
        put(fbase + (int64_t)(v_) * ns + col, f_);                                               \
        if (DIGEST) {                                                                            \
            const int64_t s_ = (sbase + (int64_t)(v_) * ns)[col];                                \
            dig += mix64(mix64((uint64_t)(v_) ^ (uint64_t)s_) ^ (uint64_t)(f_));                 \
        }                                                                                        \
    }

    // The refined passes' per-item inputs (overlap masks, one byte per scenario, or extra
    // times, four bytes), one row per walk item with this tile's 64 columns, staged in LDS
    // in [item][lane] order: half a round of rows at a time, loaded straight from memory into
    // LDS (no registers), one half ahead of its use -- the first half of a round during the
    // previous round's second half, the second half during its own first half -- so that
    // the wait for a half finds it arrived long ago.  (The arrays have a round of rows past
    // the last item.)  Only rows that overlap detection flagged as holding a nonzero value
    // are fetched (an unflagged compute item is not inflated): `want` has bit q set for
    // item q of the round.
    // Where the pass is bound by HBM -- a final pass over many scenario tiles, whose timeline
    // stores fill the memory system -- the bytes of every row count; the masks of a pass bound
    // by its chain of items (not the final one, or few tiles) are instead fetched whole, a
    // round ahead in registers (lane l: 16 bytes, row l / 4, +16 in the second half, quarter
    // l % 4), because there a second wait in the middle of a round costs more than the bytes.
    // Extra times are always fetched by flag.
    const uint4 *const mrow4 = reinterpret_cast<const uint4 *>(a.tmask + (int64_t)tile * kLanes) + (lane & 3);
    const int64_t mst4 = a.mstride / 16;
    uint4 mnx0 = make_uint4(0, 0, 0, 0), mnx1 = mnx0;
    if (REFINED && !kFlagged) {
        mnx0 = mrow4[(beg + (lane >> 2)) * mst4];
        mnx1 = mrow4[(beg + 16 + (lane >> 2)) * mst4];
    }
    constexpr int kHalf = kBlock / 2;
    const uint32_t *const erow = a.ext + (int64_t)tile * kLanes + col;
    const uint32_t *const mrow = reinterpret_cast<const uint32_t *>(a.tmask + (int64_t)tile * kLanes) + lane;
    auto stage_rows = [&](int64_t row0, int h, uint32_t want) {
        for (uint32_t m = (want >> h) & ((1u << kHalf) - 1); m; m &= m - 1) {
            const int q = __builtin_ctz(m);
            if (PRORATE) {
                __builtin_amdgcn_global_load_lds(erow + (row0 + q) * a.mstride,
                                                 fstage + (wave * kBlock + h + q) * kLanes, 4, 0, 0);
            } else if (lane < kLanes / 4) {
                // a mask row is 64 bytes: sixteen lanes load four each
                __builtin_amdgcn_global_load_lds(mrow + (row0 + q) * (a.mstride / 4),
                                                 fstage + (wave * kBlock + h + q) * (kLanes / 4), 4, 0, 0);
            }
        }
    };
    // a round's flags of its compute items: lane q < 32 holds item q's flag byte
    auto round_flags = [&](uint32_t fl, int4 items, int n) -> uint32_t {
        return (uint32_t)__ballot(lane < n && lane < 32 && fl != 0 && item_kind((uint32_t)items.y) == ECHO_COMPUTE);
    };
    auto load_flags = [&](int64_t row0) -> uint32_t {
        return lane < 32 && row0 + lane < end ? (uint32_t)a.xflag[(row0 + lane) * a.n_tiles + tile] : 0u;
    };
    uint32_t fl_now = 0, fl_next = 0;     // this round's and the next round's flag bytes
    uint32_t want = 0;                    // this round's flagged compute items
    // A compute item's staged mask (wave-uniform test: a compute op whose row was staged) is
    // read before its jitter draw, so that the LDS latency hides behind the draw, and for a
    // flagged row (some nonzero mask) the class row of the lane's slowdown table with it.  An
    // extra time is read after the draw: held across it, it took the prorating variants past
    // 128 registers, and the fewer co-resident workgroups made the largest graphs walk more
    // ranks per wavefront.
    uint32_t sm = 0, srow[kTypes] = {};
    auto staged = [&](uint32_t meta, int j) -> bool {
        return REFINED && item_kind(meta) == ECHO_COMPUTE && ((want >> j) & 1u);
    };
    auto read_staged = [&](int j, uint32_t meta) {
        if (PRORATE) return;
        sm = fst[j * kLanes + col];
        if (IN == kInMaskFlags) {
#pragma unroll
            for (int t = 0; t < kTypes; ++t) srow[t] = slow[(item_class(meta) * kTypes + t) * kLanes + lane];
        }
    };
    auto apply_staged = [&](int64_t d, uint32_t meta, int j) -> int64_t {
        if (PRORATE) return d + fst32[j * kLanes + lane];
        if (IN == kInMaskFlags) return inflate_row(d, sm, srow);
        return inflate(d, sm, slow, item_class(meta), lane);
    };
    if (kFlagged && beg < end) {
        fl_now = load_flags(beg);
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        const int n0 = end - beg < kBlock ? int(end - beg) : kBlock;
        stage_rows(beg, 0, round_flags(fl_now, nxt, n0));
    }
    for (int64_t blk0 = beg; blk0 < end; blk0 += kBlock) {
        const int4 cur = nxt;
        const int nb = end - blk0 < kBlock ? int(end - blk0) : kBlock;
        // This round's items and its first half of staged rows (fetched during the last
        // round) are settled first: a wait at their first use would also wait for the
        // fetches issued below.
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        if (REFINED && !kFlagged) {
            uint4 *const f4 = reinterpret_cast<uint4 *>(fst);
            f4[lane] = mnx0;
            f4[kLanes + lane] = mnx1;
        }
        // the round's second half of rows is fetched now, into rows the last round's second
        // half has finished with, and the next round's flags with it
        if (kFlagged) {
            want = round_flags(fl_now, cur, nb);
            if (nb > kHalf) stage_rows(blk0 + kHalf, kHalf, want);
            fl_next = load_flags(blk0 + kBlock);
        }
        nxt = blk0 + kBlock + slotl < end ? items4[2 * (blk0 + kBlock + slotl) + half] : make_int4(0, 0, 0, 0);
        if (REFINED && !kFlagged && blk0 + kBlock < end) {
            mnx0 = mrow4[(blk0 + kBlock + (lane >> 2)) * mst4];
            mnx1 = mrow4[(blk0 + kBlock + 16 + (lane >> 2)) * mst4];
        }
        if (REFINED && !kFlagged) want = ~0u;     // every row staged
        // fast flags of the round, one bit per item
        const uint64_t fast_bits = __builtin_amdgcn_read_exec() &
                                   __ballot((lane < nb) && (lane < 32) && (cur.y & kFast));
        // What a fast item needs besides its op and duration, as bits of the round taken
        // once, so that its loop reads two lanes per item instead of four: the items that
        // store a start or finish of their own (passes that do not store every one), the
        // compute items with a staged row, and whether every duration of the round fits
        // 32 bits (lane 32 + j holds the high word of item j's).
        const uint32_t need_bits = (uint32_t)(__builtin_amdgcn_read_exec() &
                                              __ballot(lane < 32 && ((uint32_t)cur.y & (kNeedS | kNeedF))));
        const uint32_t stg_bits =
            !REFINED ? 0u
            : kFlagged ? want
                       : (uint32_t)(__builtin_amdgcn_read_exec() &
                                    __ballot(lane < 32 && item_kind((uint32_t)cur.y) == ECHO_COMPUTE));
        const bool small_round =
            __builtin_amdgcn_readfirstlane((__builtin_amdgcn_read_exec() & __ballot(lane >= 32 && cur.y != 0)) == 0);
        int j = 0;
        bool second_half = false;     // the round's second half of staged rows settled
        while (j < nb) {
            if (kFlagged && j == kHalf && !second_half) {
                // the second half was fetched at the round's start; the next round's first
                // half goes into the rows the first half has finished with
                __builtin_amdgcn_s_waitcnt(kWaitVm0);
                if (blk0 + kBlock < end) {
                    const int nn = end - blk0 - kBlock < kBlock ? int(end - blk0 - kBlock) : kBlock;
                    // The next round's flags and items arrived with the wait above.  The empty asm
                    // keeps their use here: left free, the compiler computes the per-lane test
                    // where they are fetched, at the round's start, and waits for them there.
                    uint32_t fl = fl_next;
                    int4 it = nxt;
                    asm volatile("" : "+v"(fl), "+v"(it.y));
                    stage_rows(blk0 + kBlock, 0, round_flags(fl, it, nn));
                }
                second_half = true;
            }
            // a run of fast items: compute/memcpy ops right after the previous op of slot 0
            // (fast bits exist only below nb, so the run ends there at the latest; with extra
            // times it also stops where the second half begins)
            int run_end = j + (int)__builtin_ctzll(~(fast_bits >> j));
            if (kFlagged && j < kHalf && run_end > kHalf) run_end = kHalf;
            int64_t s0 = lf0;
// ALL: the pass stores every start and finish, so the items' own needs are not consulted;
// JIT: some lane draws jitter (the branch stays out of the loop); SMALL: every duration
// of the round is below 2^32 ns.  The item's metadata word, and without jitter its op, are
// read only where they are used (a staged row's class, an item's own stores).
#define FAST_RUN(ALL, JIT, SMALL)                                                                \
            for (; j < run_end; ++j) {                                                           \
                const int32_t op = ((JIT) || (ALL) || DIGEST) ? __builtin_amdgcn_readlane(cur.x, j) : 0; \
                const uint32_t dlo = (uint32_t)__builtin_amdgcn_readlane(cur.x, j + 32);         \
                const int64_t dur = (SMALL) ? (int64_t)dlo                                       \
                    : (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.y, j + 32) << 32) | dlo); \
                const bool stg = REFINED && ((stg_bits >> j) & 1u);                              \
                uint32_t meta = 0;                                                               \
                if (stg) {                                                                       \
                    if (!PRORATE) meta = (uint32_t)__builtin_amdgcn_readlane(cur.y, j);          \
                    read_staged(j, meta);                                                        \
                }                                                                                \
                int64_t d = !(JIT) ? dur : (SMALL) ? jittered32(dlo, op, jt) : jittered(dur, op, jt); \
                if (stg) d = apply_staged(d, meta, j);                                           \
                const int64_t f = s0 + d;                                                        \
                if (ALL) {                                                                       \
                    put(sbase + (int64_t)op * ns + col, s0);                                     \
                    put(fbase + (int64_t)op * ns + col, f);                                      \
                } else if ((need_bits >> j) & 1u) {                                              \
                    const int32_t sop = ((JIT) || DIGEST) ? op : __builtin_amdgcn_readlane(cur.x, j); \
                    const uint32_t nm = (uint32_t)__builtin_amdgcn_readlane(cur.y, j);           \
                    if (nm & kNeedS) put(sbase + (int64_t)sop * ns + col, s0);                   \
                    if (nm & kNeedF) put(fbase + (int64_t)sop * ns + col, f);                    \
                }                                                                                \
                if (DIGEST) dig += mix64(mix64((uint64_t)op ^ (uint64_t)s0) ^ (uint64_t)f);     \
                s0 = f;                                                                          \
            }
            if (keep) {
                // (stores every start and finish: the high word's read is not worth a variant)
                if (!any_jitter) FAST_RUN(true, false, false)
                else if (small_round) FAST_RUN(true, true, true)
                else FAST_RUN(true, true, false)
            } else {
                if (small_round) {
                    if (any_jitter) FAST_RUN(false, true, true) else FAST_RUN(false, false, true)
                } else {
                    if (any_jitter) FAST_RUN(false, true, false) else FAST_RUN(false, false, false)
                }
            }
#undef FAST_RUN
            // durations are never negative: the run's last finish is its latest time
            hi_or |= (uint32_t)((uint64_t)s0 >> 32);
            lf0 = s0;
            if (j >= nb) break;
            if (kFlagged && j == kHalf && !second_half) continue;   // settle it first
            const int32_t op = __builtin_amdgcn_readlane(cur.x, j);
            const uint32_t meta = (uint32_t)__builtin_amdgcn_readlane(cur.y, j);
            const int64_t dur = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.y, j + 32) << 32) |
                                          (uint32_t)__builtin_amdgcn_readlane(cur.x, j + 32));
            const int kind = item_kind(meta);
            const int32_t far_off = __builtin_amdgcn_readlane(cur.z, j);
            const int32_t coll = __builtin_amdgcn_readlane(cur.w, j);
            const int32_t nfar = __builtin_amdgcn_readlane(cur.z, j + 32);
            const uint32_t aux = (uint32_t)__builtin_amdgcn_readlane(cur.w, j + 32);
            const int st = item_stream(meta);
            if (kind == kResolve) {
                // a comm op's barrier, due right before its first successor
                int64_t f;
                MEET(coll, op, aux, (int32_t)dur, f, far_off)
                xmax = f > xmax ? f : xmax;
                const int sq = __builtin_amdgcn_readfirstlane((meta & kNoReg) ? kStreams : st);
                if (sq == 0) lf0 = f;
                else slot_set(sq, f);
                if (meta & kFold) lf0 = f > lf0 ? f : lf0;
                ++j;
                continue;
            }
            const unsigned mask = item_regmask(meta);
            int64_t ready = 0;
            if (mask & 1u) ready = lf0;
            for (unsigned m = mask & ~1u; m; m &= m - 1) {
                const int64_t x = slot_get(__builtin_amdgcn_readfirstlane(__builtin_ctz(m)));
                ready = x > ready ? x : ready;
            }
            for (int32_t q = 0; q < nfar; ++q) {
                const int64_t u = a.far[far_off + q];
                const int64_t fu = (fbase + u * ns)[col];
                ready = fu > ready ? fu : ready;
            }
            if ((meta | keep) & kNeedS) put(sbase + (int64_t)op * ns + col, ready);
            if (kind == ECHO_COMM) {
                // launch: publish this member's launch time, then count the arrival
                if (aux & kAuxLocal) {
                    const int ch = aux_channel(aux), par = aux_parity(aux);
                    __hip_atomic_fetch_max(&lbar[ch][par][lane], (unsigned long long)ready, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
                    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
                    if (lane == 0)
                        __hip_atomic_fetch_add(&lcnt[ch][par], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                } else if (aux & kAuxSlots) {
                    // this member's slot (its index is in the item's duration field): one store,
                    // no wait -- the value is its own arrival flag
                    if (active)
                        __hip_atomic_store(a.slots + dur * ns + sigma, ready, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                } else {
                    if (active)
                        __hip_atomic_fetch_max(a.arrive + (int64_t)coll * ns + sigma, (unsigned long long)ready,
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                    if (lane == 0)
                        __hip_atomic_fetch_add(a.count + (int64_t)coll * a.n_tiles + tile, 1u, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                }
            } else {
                const bool stg = staged(meta, j);
                if (stg) read_staged(j, meta);
                int64_t d = any_jitter ? jittered(dur, op, jt) : dur;
                if (stg) d = apply_staged(d, meta, j);
                const int64_t f = ready + d;
                hi_or |= (uint32_t)((uint64_t)f >> 32);
                if ((meta | keep) & kNeedF) put(fbase + (int64_t)op * ns + col, f);
                if (DIGEST) dig += mix64(mix64((uint64_t)op ^ (uint64_t)ready) ^ (uint64_t)f);
                xmax = f > xmax ? f : xmax;
                const int sq = __builtin_amdgcn_readfirstlane((meta & kNoReg) ? kStreams : st);
                if (sq == 0) lf0 = f;
                else slot_set(sq, f);
            }
            ++j;
        }
        fl_now = fl_next;    // loaded at the round's start, settled by the wait at its second half
    }
#undef MEET
    if (hi_or >> 30) err |= kStatusOverflow;
    if (active && err) __hip_atomic_fetch_or(a.status, err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (FINAL && active && !dead) {
        // finishes along a FIFO stream never decrease: the last op of each slot holds its
        // maximum; ops without a slot went into xmax
        int64_t smax = lf0 > xmax ? lf0 : xmax;
#pragma unroll
        for (int q = 1; q < kStreams; ++q) smax = slot_get(q) > smax ? slot_get(q) : smax;
        __hip_atomic_fetch_max(reinterpret_cast<unsigned long long *>(a.step) + sigma, (unsigned long long)smax,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (DIGEST)
            __hip_atomic_fetch_add(reinterpret_cast<unsigned long long *>(a.digest) + sigma,
                                   (unsigned long long)dig, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

using WalkKernel = void (*)(WalkArgs);
WalkKernel walk_kernel(int in, bool final_pass, bool digest) {
    // flagged mask rows only in a final pass, a digest only in a final pass
    if (!final_pass) {
        if (in == kInNone) return k_walk<kInNone, false, false>;
        return in == kInExtFlags ? k_walk<kInExtFlags, false, false> : k_walk<kInMasks, false, false>;
    }
    switch (in) {
    case kInNone: return digest ? k_walk<kInNone, true, true> : k_walk<kInNone, true, false>;
    case kInMasks: return digest ? k_walk<kInMasks, true, true> : k_walk<kInMasks, true, false>;
    case kInMaskFlags: return digest ? k_walk<kInMaskFlags, true, true> : k_walk<kInMaskFlags, true, false>;
    default: return digest ? k_walk<kInExtFlags, true, true> : k_walk<kInExtFlags, true, false>;
    }
}

// ------------------------------------------------------------------ overlap detection
// One wavefront per (rank, tile).  Compute ops of one stream run back to back,
// and so do the comm ops of one stream, so for each comm stream a cursor that
// only moves forward finds every comm op overlapping the current compute op.
// After compute op v the cursor of each comm stream sits on a comm op that ends
// after v started (at or after v finished, once v had to look at that stream:
// every later compute op of v's stream starts at or after v's finish); for the next
// compute op v', "that comm op starts at or after v' ends" proves both "no
// overlap" and "cursor stays" -- one compare per comm stream in the common
// case.  A compute op's interval is
// rebuilt rather than read: a chained op starts where the previous compute op
// of its stream finished, and every finish is start + base duration (the same
// jitter draw as the composer pass, inflated by the factor that pass used);
// only unchained ops read their start.
// Factor of a class-cls compute op overlapping the collective types in mask m:
// the largest entry of the scenario's table row over them, 65536 for none.
__device__ __forceinline__ uint32_t factor_of(uint32_t m, const uint32_t *slow, int cls) {
    uint32_t F = 65536u;
    for (int t = 0; t < kTypes; ++t)
        if ((m >> t) & 1u) {
            const uint32_t x = slow[cls * kTypes + t];
            F = x > F ? x : F;
        }
    return F;
}

// Factor predicted by the tree ensemble for a compute op (class cls, base
// duration d0) overlapped by the collective types in mask m (Sec. 6): for each
// type, the base score plus one leaf per tree, kept inside [65536, 2^20); the
// largest over the types.  Trees are walked from device memory (the walk stops at
// a leaf; paths are at most ECHO_TREE_DEPTH splits long): when every lane that
// needs a type shares one feature vector, once for the wavefront with one tree
// per lane, else per lane.
constexpr int kForestLanes = 16;
constexpr int kPre = 8;          // unchained starts prefetched per round of overlap detection
constexpr int kIdStage = 1024;   // comm ops of a rank whose ids overlap detection keeps in LDS

// feat: this wavefront's LDS feature rows, feature k of lane l at feat[k * 64 + l].
__device__ uint32_t forest_factor(const OverlapArgs &a, uint32_t m, const int64_t *smax, const int32_t *nmax,
                                  int cls, int64_t d0, const echo_scenario *sc, int64_t *feat, bool knobs_uniform,
                                  int lane) {
    const int64_t *met = a.class_metrics + cls * kClassMetrics;
    feat[0 * kLanes + lane] = cls;
    feat[1 * kLanes + lane] = d0;
    feat[5 * kLanes + lane] = sc->ar_algo;
    feat[6 * kLanes + lane] = sc->bw_intra_MBps;
    feat[7 * kLanes + lane] = sc->bw_inter_MBps;
#pragma unroll
    for (int k = 0; k < kClassMetrics; ++k) feat[(8 + k) * kLanes + lane] = met[k];
    uint32_t best = 65536u;
#pragma unroll
    for (int t = 0; t < kTypes; ++t) {
        const bool has = (m >> t) & 1u;
        const uint64_t lanes_t = __ballot(has);
        if (!lanes_t) continue;
        feat[2 * kLanes + lane] = t;
        feat[3 * kLanes + lane] = smax[t];
        feat[4 * kLanes + lane] = nmax[t];
        const int first = __builtin_ctzll(lanes_t);
        const int64_t s0 = __shfl(smax[t], first);
        const int32_t n0 = __shfl(nmax[t], first);
        const bool uniform = knobs_uniform && __ballot(has && (smax[t] != s0 || nmax[t] != n0)) == 0;
        int64_t sum = a.forest_base;
        if (uniform) {
            // every lane that needs type t has lane `first`'s feature vector: the trees are
            // walked side by side, one per lane, and their leaves summed across the wavefront
            for (int32_t tr0 = 0; tr0 < a.n_trees; tr0 += kLanes) {
                const bool live = tr0 + lane < a.n_trees;
                int32_t idx = a.forest_roots[live ? tr0 + lane : 0];
                for (int step = 0; step < ECHO_TREE_DEPTH; ++step) {
                    const int4 nd = reinterpret_cast<const int4 *>(a.forest_nodes)[idx];
                    const int64_t x = feat[nd.z * kLanes + first];
                    const int64_t thr = (int64_t)(((uint64_t)(uint32_t)nd.y << 32) | (uint32_t)nd.x);
                    idx = nd.w + (x < thr ? 0 : 1);
                }
                int64_t leaf = live ? (int64_t)a.forest_leaf[idx] : 0;
#pragma unroll
                for (int o = kLanes / 2; o > 0; o >>= 1) leaf += __shfl_xor(leaf, o);
                sum += leaf;
            }
        } else {
            // kForestLanes trees walked side by side: their node loads are independent
            for (int32_t tr0 = 0; tr0 < a.n_trees; tr0 += kForestLanes) {
                int32_t idx[kForestLanes];
                bool live[kForestLanes];
#pragma unroll
                for (int q = 0; q < kForestLanes; ++q) {
                    live[q] = tr0 + q < a.n_trees;
                    idx[q] = live[q] ? a.forest_roots[tr0 + q] : 0;
                }
                // every path has at most ECHO_TREE_DEPTH splits and a leaf loops to itself, so
                // after that many steps each walk rests on its leaf: no per-lane exit
                for (int step = 0; step < ECHO_TREE_DEPTH; ++step) {
                    int4 nd[kForestLanes];          // threshold low, threshold high, feature, left
#pragma unroll
                    for (int q = 0; q < kForestLanes; ++q)
                        nd[q] = reinterpret_cast<const int4 *>(a.forest_nodes)[idx[q]];
#pragma unroll
                    for (int q = 0; q < kForestLanes; ++q) {
                        const int64_t x = feat[nd[q].z * kLanes + lane];
                        const int64_t thr = (int64_t)(((uint64_t)(uint32_t)nd[q].y << 32) | (uint32_t)nd[q].x);
                        idx[q] = nd[q].w + (x < thr ? 0 : 1);
                    }
                }
#pragma unroll
                for (int q = 0; q < kForestLanes; ++q)
                    if (live[q]) sum += a.forest_leaf[idx[q]];
            }
        }
        sum = sum < 65536 ? 65536 : sum;
        sum = sum >= (int64_t(1) << 20) ? (int64_t(1) << 20) - 1 : sum;
        if (has) best = (uint32_t)sum > best ? (uint32_t)sum : best;
    }
    return best;
}

// ---- compact ensemble (LDS): features compared by bin (see CompactForest)
// Bin of x for a feature with sorted thresholds T[0..n): how many are <= x.
__device__ __forceinline__ int32_t fx_bin(const int64_t *T, int32_t n, int64_t x) {
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (T[mid] <= x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Bins of every collective's S and cost N (features 3 and 4) and of every compute
// record's base duration (feature 1).
__global__ void k_forest_bins(CollTable colls, const ComputeRec *cp, int64_t n_cp, CompactForest fx) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    const int64_t *T1 = fx.thr + fx.thr_off[1], *T3 = fx.thr + fx.thr_off[3], *T4 = fx.thr + fx.thr_off[4];
    const int32_t n1 = fx.thr_off[2] - fx.thr_off[1], n3 = fx.thr_off[4] - fx.thr_off[3],
                  n4 = fx.thr_off[5] - fx.thr_off[4];
    for (int64_t c = tid; c < colls.n; c += nth) {
        fx.coll_bin[2 * c] = fx_bin(T3, n3, colls.bytes[c]);
        fx.coll_bin[2 * c + 1] = fx_bin(T4, n4, colls.N[c]);
    }
    for (int64_t i = tid; i < n_cp; i += nth) fx.cp_bin[i] = fx_bin(T1, n1, cp[i].dur);
}

// Ensemble prediction from the compact LDS form, for the collective types in mask m
// (per lane), as forest_factor computes it.  fb: this wavefront's bin rows in LDS,
// feature f of lane l at fb[f * 64 + l] (rows 5-7: the scenario's knobs, set once;
// rows 12-15: 0).  bS/bN: per type, the largest bins of S and N among the overlapping
// type-t comm ops.  When every lane that has type t in its mask shares its feature
// vector (knobs_uniform and equal S and N bins), the trees are walked once for the
// wavefront, one tree per lane; otherwise each lane walks every tree on its own path.
__device__ uint32_t forest_factor_compact(const OverlapArgs &a, uint32_t m, const int32_t *bS, const int32_t *bN,
                                          int cls, int32_t bd0, const uint32_t *fw, const int32_t *froots, uint16_t *fb,
                                          bool knobs_uniform, int lane) {
    const int32_t *cb = a.fx.cbin + cls * kFxFeatures;
    fb[0 * kLanes + lane] = (uint16_t)cb[0];
    fb[1 * kLanes + lane] = (uint16_t)bd0;
#pragma unroll
    for (int k = 8; k < kFxFeatures; ++k) fb[k * kLanes + lane] = (uint16_t)cb[k];
    uint32_t best = 65536u;
#pragma unroll
    for (int t = 0; t < kTypes; ++t) {
        const bool has = (m >> t) & 1u;
        const uint64_t lanes_t = __ballot(has);
        if (!lanes_t) continue;
        fb[2 * kLanes + lane] = (uint16_t)a.fx.tbin[t];
        fb[3 * kLanes + lane] = (uint16_t)bS[t];
        fb[4 * kLanes + lane] = (uint16_t)bN[t];
        const int first = __builtin_ctzll(lanes_t);
        const int32_t s0 = __builtin_amdgcn_readlane(bS[t], first), n0 = __builtin_amdgcn_readlane(bN[t], first);
        const bool uniform = knobs_uniform && __ballot(has && (bS[t] != s0 || bN[t] != n0)) == 0;
        int64_t sum = a.forest_base;
        if (uniform) {
            // One feature vector (lane `first`'s) for every lane that needs type t: the
            // trees are walked side by side, one per lane, and their leaves summed across
            // the wavefront.
            for (int32_t tr0 = 0; tr0 < a.n_trees; tr0 += kLanes) {
                const bool live = tr0 + lane < a.n_trees;
                int32_t idx = froots[live ? tr0 + lane : 0];
                for (int step = 0; step < ECHO_TREE_DEPTH; ++step) {
                    const uint32_t w = fw[idx];
                    const uint32_t f = w & 15u;
                    const uint32_t r = (w >> 4) & ((1u << kFxRankBits) - 1);
                    const int32_t off = f == kFxLeaf ? 0 : (int32_t)(w >> (4 + kFxRankBits));
                    const uint32_t x = fb[f * kLanes + first];
                    idx += off + (x > r ? 1 : 0);
                }
                int64_t leaf = live ? (int64_t)((int32_t)fw[idx] >> 4) : 0;
#pragma unroll
                for (int o = kLanes / 2; o > 0; o >>= 1) leaf += __shfl_xor(leaf, o);
                sum += leaf;
            }
        } else {
            for (int32_t tr0 = 0; tr0 < a.n_trees; tr0 += kForestLanes) {
                int32_t idx[kForestLanes];
                bool live[kForestLanes];
#pragma unroll
                for (int q = 0; q < kForestLanes; ++q) {
                    live[q] = tr0 + q < a.n_trees;
                    idx[q] = froots[live[q] ? tr0 + q : 0];
                }
                for (int step = 0; step < ECHO_TREE_DEPTH; ++step) {
                    uint32_t w[kForestLanes];
#pragma unroll
                    for (int q = 0; q < kForestLanes; ++q) w[q] = fw[idx[q]];
#pragma unroll
                    for (int q = 0; q < kForestLanes; ++q) {
                        const uint32_t f = w[q] & 15u;
                        const uint32_t r = (w[q] >> 4) & ((1u << kFxRankBits) - 1);
                        const int32_t off = f == kFxLeaf ? 0 : (int32_t)(w[q] >> (4 + kFxRankBits));
                        const uint32_t x = fb[f * kLanes + lane];
                        idx[q] += off + (x > r ? 1 : 0);
                    }
                }
#pragma unroll
                for (int q = 0; q < kForestLanes; ++q)
                    if (live[q]) sum += (int32_t)fw[idx[q]] >> 4;
            }
        }
        sum = sum < 65536 ? 65536 : sum;
        sum = sum >= (int64_t(1) << 20) ? (int64_t(1) << 20) - 1 : sum;
        if (has) best = (uint32_t)sum > best ? (uint32_t)sum : best;
    }
    return best;
}

// PRORATE: also measure o, the part of [s_v, f_v) covered by the union of the
// overlapping comm intervals (a merge of the per-stream interval lists in start
// order), and record the extra time q16(min(o, D), F) - min(o, D) instead of a mask.
// DETECT: flag the scenarios whose durations change (fixed-point iteration).
// FOREST: the factor is the tree ensemble's prediction (recorded as an extra time):
// 1 walks the ensemble from device memory, 2 from its compact form in LDS (a workgroup
// of kFxWaves wavefronts, one (rank, tile) each, shares one copy of the nodes).
// NC: room for this many comm streams per rank (the cursor and merge state scale with it).
constexpr int kFxWaves = 4;
// The fixed-point prorating variant with four comm streams is held to four waves per SIMD
// (at most 128 registers; left free it took 142, three waves per SIMD, and its 4,096
// wavefronts on the 1024-rank workload ran in two rounds): a few spilled registers cost far
// less than the second round.
template <bool PRORATE, bool DETECT, int FOREST, int NC>
__global__ __launch_bounds__(64 * (FOREST == 2 ? kFxWaves : 1))
__attribute__((amdgpu_waves_per_eu(PRORATE && DETECT && FOREST == 0 && NC == 4 ? 4 : 1))) void k_overlap(OverlapArgs a) {
    constexpr bool EXT = PRORATE || FOREST != 0;  // output: extra time per op instead of a mask
    constexpr int W = FOREST == 2 ? kFxWaves : 1;      // wavefronts per workgroup
    constexpr int STAGE = FOREST == 2 ? kIdStage / 4 : kIdStage;
    // unchained starts prefetched per round: as many as the registers allow while the
    // variants with four comm streams keep four wavefronts per SIMD (the prorating and
    // fixed-point variants hold more state for their block checks and interval merges)
    constexpr int NPRE = FOREST ? kPre : PRORATE ? kPre / 4 : DETECT ? (NC == 4 ? kPre / 2 : kPre / 4) : NC == 4 ? kPre : kPre / 2;
    __shared__ int64_t feat[FOREST == 1 ? 12 * kLanes : 1];   // the ensemble's feature vectors, one per lane
    __shared__ uint16_t fbin[FOREST == 2 ? W * kFxRows * kLanes : 1];   // compact: bin rows per lane
    extern __shared__ uint32_t fwords[];         // compact: the ensemble's nodes
    __shared__ int32_t sid_all[W * STAGE];       // the rank's comm op ids and collective types, staged
    __shared__ uint8_t stype_all[W * STAGE];
    // masks of the round's ops, [op][lane]: written out row by row once per round
    __shared__ __align__(16) uint8_t mstage[EXT ? 16 : kLanes * kLanes];
    if (a.stable && __builtin_amdgcn_readfirstlane(__hip_atomic_load(a.stable, __ATOMIC_RELAXED,
                                                                      __HIP_MEMORY_SCOPE_AGENT)))
        return;                                  // every scenario is at its fixed point
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t unit = (int64_t)blockIdx.x * W + wave;       // (rank, tile) of this wavefront
    const bool valid = unit < (int64_t)a.n_ranks * a.n_tiles;
    const int32_t r = valid ? (int32_t)(unit / a.n_tiles) : 0;
    const int32_t tile = valid ? (int32_t)(unit % a.n_tiles) : 0;
    int32_t *const sid = sid_all + wave * STAGE;
    uint8_t *const stype = stype_all + wave * STAGE;
    if (FOREST == 2) {
        // the nodes, then the roots of the trees
        for (int i = threadIdx.x; i < a.fx.n_words; i += 64 * W) fwords[i] = a.fx.words[i];
        for (int i = threadIdx.x; i < a.n_trees; i += 64 * W) fwords[a.fx.n_words + i] = (uint32_t)a.forest_roots[i];
    }
    const bool active = tile * kLanes + lane < a.n_scen;
    const int32_t col = active ? lane : a.n_scen - 1 - tile * kLanes;
    const int32_t sigma = tile * kLanes + col;
    const int64_t ns = a.n_scen;
    const int64_t *const sbase = a.start + (int64_t)tile * kLanes;
    const int64_t *const fbase = a.finish + (int64_t)tile * kLanes;
    uint8_t *const obase = a.tmask + (int64_t)tile * kLanes;
    uint32_t *const ebase = a.ext + (int64_t)tile * kLanes;
    const echo_scenario *sc = a.scen + sigma;
    const uint32_t *slow = &sc->slowdown_q16[0][0];
    const int32_t amp = sc->jitter_amp_q16;
    const Jitter jt = make_jitter(sc->jitter_seed, sc->jitter_stream, amp);
    // one branch for the wavefront: a lane without jitter draws the identity factor
    const bool any_jitter = __builtin_amdgcn_readfirstlane(__ballot(amp != 0) != 0);
    const int64_t *cl_off = a.cl_off + (int64_t)r * kStreams;
    const int64_t *cp_off = a.cp_off + (int64_t)r * kStreams;
    bool changed = false;                        // some duration differs from the previous pass's
    bool ext_over = false;                       // a prorated extra time does not fit 32 bits

    // Stage the rank's comm lists in LDS: a cursor move then costs one memory round trip
    // (the comm op's interval) instead of two (its id, then the interval).
    const int64_t cbase = cl_off[0];
    const int64_t nstage = !valid ? 0 : cl_off[kStreams] - cbase < STAGE ? cl_off[kStreams] - cbase : STAGE;
    for (int64_t i = lane; i < nstage; i += kLanes) {
        sid[i] = a.cl[cbase + i];
        stype[i] = a.cl_type[cbase + i];
    }
    __syncthreads();
    if (!valid) return;                          // past the last (rank, tile); after the shared fill
    // compact ensemble: this wavefront's bin rows; the scenario knobs' rows are fixed
    uint16_t *const fb = fbin + (FOREST == 2 ? wave * kFxRows * kLanes : 0);
    bool knobs_uniform = false;
    if (FOREST == 2) {
        const int32_t k5 = fx_bin(a.fx.thr + a.fx.thr_off[5], a.fx.thr_off[6] - a.fx.thr_off[5], sc->ar_algo);
        const int32_t k6 = fx_bin(a.fx.thr + a.fx.thr_off[6], a.fx.thr_off[7] - a.fx.thr_off[6], sc->bw_intra_MBps);
        const int32_t k7 = fx_bin(a.fx.thr + a.fx.thr_off[7], a.fx.thr_off[8] - a.fx.thr_off[7], sc->bw_inter_MBps);
        fb[5 * kLanes + lane] = (uint16_t)k5;
        fb[6 * kLanes + lane] = (uint16_t)k6;
        fb[7 * kLanes + lane] = (uint16_t)k7;
#pragma unroll
        for (int k = kFxFeatures; k < kFxRows; ++k) fb[k * kLanes + lane] = 0;
        knobs_uniform = __ballot(k5 != __builtin_amdgcn_readfirstlane(k5) || k6 != __builtin_amdgcn_readfirstlane(k6) ||
                                 k7 != __builtin_amdgcn_readfirstlane(k7)) == 0;
    } else if (FOREST == 1) {
        const int64_t k6 = sc->bw_intra_MBps, k7 = sc->bw_inter_MBps;
        const int32_t k5 = sc->ar_algo;
        knobs_uniform = __ballot(k5 != __builtin_amdgcn_readfirstlane(k5) || k6 != __shfl(k6, 0) ||
                                 k7 != __shfl(k7, 0)) == 0;
    }
    // comm op at position x of the rank's lists and its collective type
    auto comm_id = [&](int64_t x) -> int64_t {
        const int64_t o = x - cbase;
        if (o < nstage) return sid[o];
        return __hip_atomic_load(a.cl + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    auto comm_type = [&](int64_t x) -> uint32_t {
        const int64_t o = x - cbase;
        if (o < nstage) return stype[o];
        // an atomic load keeps this read and the LDS one from merging into a flat load
        return __hip_atomic_load(a.cl_type + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };

    // comm streams of this rank that carry comm ops, packed to the front
    int64_t kb[NC];
    int32_t nk[NC];
    int ncs = 0;
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        kb[k] = 0;
        nk[k] = 0;
    }
    for (int k = 0; k < kStreams; ++k) {
        const int64_t b = cl_off[k], n = cl_off[k + 1] - b;
        if (n == 0) continue;
#pragma unroll
        for (int q = 0; q < NC; ++q)
            if (q == ncs) {
                kb[q] = b;
                nk[q] = (int32_t)n;
            }
        ++ncs;
    }
    if (ncs > NC) {
        // more comm streams than this variant holds: the loader counts them, so never
        if (lane == 0) __hip_atomic_fetch_or(a.status, kStatusRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }

    for (int s = 0; s < kStreams; ++s) {
        const int64_t b0 = cp_off[s], b1 = cp_off[s + 1];
        if (b0 == b1) continue;
        int32_t p[NC];
        int64_t cs[NC], cf[NC];
#pragma unroll
        for (int k = 0; k < NC; ++k) {
            p[k] = 0;
            cs[k] = kInf;
            cf[k] = kInf;
            if (k < ncs) {
                const int64_t c = a.cl[kb[k]];
                cs[k] = (sbase + c * ns)[col];
                cf[k] = (fbase + c * ns)[col];
            }
        }
        // earliest start among the cursors: an op ending by then overlaps nothing
        int64_t cmin = kInf;
#pragma unroll
        for (int k = 0; k < NC; ++k) cmin = cs[k] < cmin ? cs[k] : cmin;
        int64_t fprev = 0;
        // lane j holds compute record i0 + j of the current round of 64
        const int4 *recs = reinterpret_cast<const int4 *>(a.cp);
        int4 nxt = b0 + lane < b1 ? recs[b0 + lane] : make_int4(0, 0, 0, 0);
        int32_t nxt_pos = b0 + lane < b1 ? a.cp_pos[b0 + lane] : 0;
        for (int64_t i0 = b0; i0 < b1; i0 += kLanes) {
            const int4 cur = nxt;
            const int32_t cur_pos = nxt_pos;
            // settle the round's records here, once, so the per-op loop below carries
            // no memory wait (a wait there would also wait for the previous op's store)
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
            nxt = i0 + kLanes + lane < b1 ? recs[i0 + kLanes + lane] : make_int4(0, 0, 0, 0);
            nxt_pos = i0 + kLanes + lane < b1 ? a.cp_pos[i0 + kLanes + lane] : 0;
            const int nr = b1 - i0 < kLanes ? int(b1 - i0) : kLanes;
            // the starts of the round's first NPRE unchained ops, fetched together
            const uint64_t unchained = __builtin_amdgcn_read_exec() &
                                       __ballot(lane < nr && !((uint32_t)cur.y & kChained));
            int64_t pre[NPRE];
            // finishes of the round's blocks' last ops (stored by the walk): a block ending
            // before every cursor starts is skipped whole
            constexpr int kBlocks = kLanes / kOverlapBlock;
            int64_t ck[kBlocks];
            // the fixed-point variants (every pass after the first reads the previous pass's
            // values): the current block's previous masks or extra times
            uint32_t old8[DETECT ? kOverlapBlock : 1];
#pragma unroll
            for (int b = 0; b < kBlocks; ++b) {
                ck[b] = kInf;
                if (b * kOverlapBlock < nr) {
                    const int jl = (b + 1) * kOverlapBlock - 1 < nr ? (b + 1) * kOverlapBlock - 1 : nr - 1;
                    const int64_t vl = __builtin_amdgcn_readlane(cur.x, jl);
                    ck[b] = (fbase + vl * ns)[col];
                }
            }
            {
                uint64_t um = unchained;
#pragma unroll
                for (int q = 0; q < NPRE; ++q) {
                    pre[q] = 0;
                    if (um) {
                        const int jq = __builtin_ctzll(um);
                        um &= um - 1;
                        const int64_t vq = __builtin_amdgcn_readlane(cur.x, jq);
                        pre[q] = (sbase + vq * ns)[col];
                    }
                }
                __builtin_amdgcn_s_waitcnt(kWaitVm0);
            }
            for (int j = 0; j < nr; ++j) {
                if ((j & (kOverlapBlock - 1)) == 0) {
                    if (DETECT && a.prev_refined) {
                        // the previous pass's masks (extra times) of the block's ops, fetched
                        // together: one memory round trip per block instead of one per op
#pragma unroll
                        for (int q = 0; q < kOverlapBlock; ++q) {
                            old8[q] = 0;
                            if (j + q < nr) {
                                const int64_t rq = (int64_t)__builtin_amdgcn_readlane(cur_pos, j + q) * a.mstride;
                                old8[q] = EXT ? (ebase + rq)[col] : (uint32_t)(obase + rq)[col];
                            }
                        }
                        __builtin_amdgcn_s_waitcnt(kWaitVm0);
                    }
                    int64_t c = kInf;
#pragma unroll
                    for (int b = 0; b < kBlocks; ++b)
                        if (b == (j >> 3)) c = ck[b];
                    if (!__builtin_amdgcn_readfirstlane(__ballot(c > cmin) != 0)) {
                        // every op of the block ends by cmin: no overlaps, no cursor moves
                        const int je = j + kOverlapBlock < nr ? j + kOverlapBlock : nr;
                        if (EXT) {
                            // no extra times; DETECT: a duration changes where the previous
                            // pass added one
                            if (DETECT && a.prev_refined) {
                                uint32_t eo = 0;
#pragma unroll
                                for (int q = 0; q < kOverlapBlock; ++q) eo |= old8[q];
                                changed |= eo != 0;
                            }
                            for (int jj = j; jj < je; ++jj)
                                (ebase + (int64_t)__builtin_amdgcn_readlane(cur_pos, jj) * a.mstride)[col] = 0;
                        } else {
                            for (int jj = j; jj < je; ++jj) mstage[jj * kLanes + lane] = 0;
                            if (DETECT && a.prev_refined) {
                                // an op inflated in the previous pass runs with D now: a change
                                // unless its factor left D as it was
                                const uint32_t *const mo = old8;
#pragma unroll
                                for (int q = 0; q < kOverlapBlock; ++q) {
                                    if (!__builtin_amdgcn_readfirstlane(__ballot(mo[q] != 0) != 0)) continue;
                                    const int64_t vq = __builtin_amdgcn_readlane(cur.x, j + q);
                                    const int mq = __builtin_amdgcn_readlane(cur.y, j + q);
                                    const int64_t dq = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.w, j + q) << 32) |
                                                                 (uint32_t)__builtin_amdgcn_readlane(cur.z, j + q));
                                    const int64_t Dq = any_jitter ? jittered(dq, (int32_t)vq, jt) : dq;
                                    if (mo[q] != 0) changed |= q16(Dq, factor_of(mo[q], slow, mq & 7)) != Dq;
                                }
                            }
                        }
                        fprev = c;
                        j = je - 1;
                        continue;
                    }
                }
                const int64_t v = __builtin_amdgcn_readlane(cur.x, j);
                // v's row of the per-item outputs (computed where used: the common path needs none)
                auto row = [&]() { return (int64_t)__builtin_amdgcn_readlane(cur_pos, j) * a.mstride; };
                const int meta = __builtin_amdgcn_readlane(cur.y, j);
                const int cls = meta & 7;
                const int64_t d0 = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(cur.w, j) << 32) |
                                             (uint32_t)__builtin_amdgcn_readlane(cur.z, j));
                // Loads in this loop are waited for on their own path (explicit vmcnt(0)):
                // left pending, they would make the compiler wait at the next join, on
                // every path, for the previous op's store as well.
                int64_t sv = fprev;
                if (__builtin_expect(!(meta & kChained), 0)) {
                    const int ord = __builtin_popcountll(unchained & ((uint64_t(1) << j) - 1));
                    if (ord < NPRE) {
#pragma unroll
                        for (int q = 0; q < NPRE; ++q)
                            if (q == ord) sv = pre[q];
                    } else {
                        sv = (sbase + v * ns)[col];
                        __builtin_amdgcn_s_waitcnt(kWaitVm0);
                    }
                }
                const int64_t D = any_jitter ? jittered(d0, (int32_t)v, jt) : d0;
                int64_t d = D;                   // the duration v ran with in the previous pass
                uint32_t m_old = 0, e_old = 0;
                if (a.prev_refined) {
                    uint32_t ov = 0;
                    if (DETECT) {
#pragma unroll
                        for (int q = 0; q < kOverlapBlock; ++q)
                            if (q == (j & (kOverlapBlock - 1))) ov = old8[q];
                    } else {
                        ov = EXT ? (ebase + row())[col] : (uint32_t)(obase + row())[col];
                        __builtin_amdgcn_s_waitcnt(kWaitVm0);
                    }
                    if (EXT) {
                        e_old = ov;
                        d = D + e_old;
                    } else {
                        m_old = ov;
                        if (m_old != 0) d = q16(D, factor_of(m_old, slow, cls));
                    }
                }
                const int64_t fv = sv + d;
                fprev = fv;
                const bool busy = cmin < fv;
                uint32_t m = 0;                            // types of the comm ops overlapping v
                int64_t o = 0;                             // covered length (PRORATE)
                int64_t smax[kTypes];                      // FOREST: largest S per overlapping type
                int32_t nmax[kTypes];                      //         and most members (compact: their bins)
    #pragma unroll
                for (int tt = 0; tt < kTypes; ++tt) {
                    smax[tt] = 0;
                    nmax[tt] = 0;
                }
// note the comm op at list position x_ (type ty_) among v's overlaps, for the ensemble's features
#define NOTE_FOREST(x_, ty_)                                                                     \
    if (FOREST) {                                                                                \
        const int32_t cc_ = a.cl_coll[x_];                                                       \
        const int64_t S_ = FOREST == 2 ? a.fx.coll_bin[2 * cc_] : a.coll_bytes[cc_];            \
        const int32_t N_ = FOREST == 2 ? a.fx.coll_bin[2 * cc_ + 1] : a.coll_N[cc_];            \
        _Pragma("unroll") for (int tt = 0; tt < kTypes; ++tt) if (tt == (int)(ty_)) {            \
            smax[tt] = S_ > smax[tt] ? S_ : smax[tt];                                            \
            nmax[tt] = N_ > nmax[tt] ? N_ : nmax[tt];                                            \
        }                                                                                        \
    }
                if (busy) {
    #pragma unroll
                    for (int k = 0; k < NC; ++k) {
                        if (k >= ncs) break;
                        if (!(cs[k] < fv)) continue;
                        if (!PRORATE) {
                            // The cursor walks the intervals that start before v ends; one
                            // that also ends before then is behind every later op of this
                            // compute stream (each starts at or after v's finish) and is
                            // passed for good, so every comm interval is loaded once, when the
                            // cursor reaches it.
                            while (cs[k] < fv) {
                                const int64_t lo = sv > cs[k] ? sv : cs[k], hi = fv < cf[k] ? fv : cf[k];
                                if (lo < hi) {
                                    const uint32_t ty = comm_type(kb[k] + p[k]);
                                    m |= 1u << ty;
                                    NOTE_FOREST(kb[k] + p[k], ty)
                                }
                                if (cf[k] >= fv) break;    // reaches v's end: later ops may overlap it
                                ++p[k];
                                if (p[k] < nk[k]) {
                                    const int64_t c = comm_id(kb[k] + p[k]);
                                    cs[k] = (sbase + c * ns)[col];
                                    cf[k] = (fbase + c * ns)[col];
                                } else {
                                    cs[k] = kInf;
                                    cf[k] = kInf;
                                }
                            }
                            continue;
                        }
                        while (cf[k] <= sv) {              // ends before v starts: never again
                            ++p[k];
                            if (p[k] < nk[k]) {
                                const int64_t c = comm_id(kb[k] + p[k]);
                                cs[k] = (sbase + c * ns)[col];
                                cf[k] = (fbase + c * ns)[col];
                            } else {
                                cs[k] = kInf;
                                cf[k] = kInf;
                            }
                        }
                    }
                    if (PRORATE) {
                        // merge the streams' overlapping intervals in start order; every one of
                        // them ends after sv (each stream's intervals are disjoint and sorted)
                        int32_t q[NC];
                        int64_t qs[NC], qf[NC];
    #pragma unroll
                        for (int k = 0; k < NC; ++k) {
                            q[k] = p[k];
                            qs[k] = k < ncs ? cs[k] : kInf;
                            qf[k] = k < ncs ? cf[k] : kInf;
                        }
                        int64_t t = sv;                    // covered up to here
                        for (;;) {
                            int bk = -1;
                            int64_t bs = fv;
    #pragma unroll
                            for (int k = 0; k < NC; ++k)
                                if (qs[k] < bs) {
                                    bs = qs[k];
                                    bk = k;
                                }
                            if (bk < 0) break;
    #pragma unroll
                            for (int k = 0; k < NC; ++k) {
                                if (k != bk) continue;
                                const int64_t lo = sv > qs[k] ? sv : qs[k], hi = fv < qf[k] ? fv : qf[k];
                                if (lo < hi) {
                                    const uint32_t ty = comm_type(kb[k] + q[k]);
                                    m |= 1u << ty;
                                    NOTE_FOREST(kb[k] + q[k], ty)
                                    const int64_t from = lo > t ? lo : t;
                                    if (hi > from) {
                                        o += hi - from;
                                        t = hi;
                                    }
                                }
                                if (++q[k] < nk[k]) {
                                    const int64_t c = comm_id(kb[k] + q[k]);
                                    qs[k] = (sbase + c * ns)[col];
                                    qf[k] = (fbase + c * ns)[col];
                                    __builtin_amdgcn_s_waitcnt(kWaitVm0);
                                } else {
                                    qs[k] = kInf;
                                }
                            }
                        }
                    }
                    __builtin_amdgcn_s_waitcnt(kWaitVm0);
                    cmin = kInf;
#pragma unroll
                    for (int k = 0; k < NC; ++k) cmin = cs[k] < cmin ? cs[k] : cmin;
                }
#undef NOTE_FOREST
                if (EXT) {
                    uint32_t e = 0;
                    if (m != 0) {
                        uint32_t F;
                        if (FOREST == 2) {
                            int32_t bS[kTypes];
#pragma unroll
                            for (int tt = 0; tt < kTypes; ++tt) bS[tt] = (int32_t)smax[tt];
                            const int32_t bd0 = a.fx.cp_bin[i0 + j];
                            F = forest_factor_compact(a, m, bS, nmax, cls, bd0, fwords,
                                                      reinterpret_cast<const int32_t *>(fwords) + a.fx.n_words, fb,
                                                      knobs_uniform, lane);
                        } else if (FOREST == 1) {
                            F = forest_factor(a, m, smax, nmax, cls, d0, sc, feat, knobs_uniform, lane);
                        } else {
                            F = factor_of(m, slow, cls);
                        }
                        const int64_t oc = PRORATE ? (o < D ? o : D) : D;
                        const int64_t x = q16(oc, F) - oc;
                        ext_over |= x >= (int64_t)kExtLimit;
                        e = x >= (int64_t)kExtLimit ? kExtLimit : (uint32_t)x;
                    }
                    if (DETECT) changed |= e != e_old;
                    (ebase + row())[col] = e;
                    // flag the row (the walk fetches only flagged rows); flags are cleared once
                    // per compose and only ever set, so a row flagged by an earlier refinement
                    // whose extra times are zero now is fetched and adds zero
                    if (__builtin_amdgcn_readfirstlane(__ballot(e != 0) != 0) && lane == 0)
                        a.xflag[(int64_t)__builtin_amdgcn_readlane(cur_pos, j) * a.n_tiles + tile] = 1;
                } else {
                    if (DETECT && m != m_old)
                        changed |= (m == 0 ? D : q16(D, factor_of(m, slow, cls))) != d;
                    mstage[j * kLanes + lane] = (uint8_t)m;
                }
            }
            if (!EXT && lane < nr) {
                // lane L writes the 64 masks of the round's op L to that op's row, and the
                // row's flag: whether any of them is nonzero (the walk fetches only those rows)
                const uint4 *const src = reinterpret_cast<const uint4 *>(mstage + lane * kLanes);
                uint4 *const dst = reinterpret_cast<uint4 *>(obase + (int64_t)cur_pos * a.mstride);
                uint32_t any = 0;
#pragma unroll
                for (int q = 0; q < kLanes / 16; ++q) {
                    const uint4 v = src[q];
                    dst[q] = v;
                    any |= v.x | v.y | v.z | v.w;
                }
                a.xflag[(int64_t)cur_pos * a.n_tiles + tile] = any != 0;
            }
        }
    }
    if (DETECT && active && changed)
        __hip_atomic_fetch_or(a.chg + sigma, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (active && ext_over) __hip_atomic_fetch_or(a.status, kStatusRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Count the refinement of each scenario whose durations changed; flag stability.
__global__ __launch_bounds__(256) void k_settle(unsigned *chg, int32_t n_scen, int32_t *refinements,
                                                 unsigned *stable) {
    int any = 0;
    for (int32_t i = threadIdx.x; i < n_scen; i += blockDim.x) {
        if (chg[i]) {
            any = 1;
            if (refinements) refinements[i] += 1;
            chg[i] = 0;
        }
    }
    any = __syncthreads_or(any);
    if (threadIdx.x == 0 && !any) *stable = 1u;
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
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
                       int64_t *slots, int64_t n_slot_values, int64_t *step, uint64_t *digest, hipStream_t stream) {
    int64_t n = std::max<int64_t>(std::max(n_arrive, n_count), n_slot_values);
    if (n_scen > n) n = n_scen;
    hipLaunchKernelGGL(k_init, dim3(grid_for(n, 256)), dim3(256), 0, stream, scen, n_scen, arrive,
                       n_arrive, count, n_count, slots, n_slot_values, step, digest, g.n_cc_tables, g.status);
    return hipGetLastError();
}

hipError_t launch_clear(unsigned long long *arrive, int64_t n_arrive, unsigned *count, int64_t n_count,
                        int64_t *slots, int64_t n_slot_values, hipStream_t stream) {
    const int64_t n = std::max<int64_t>(std::max(n_arrive, n_count), n_slot_values);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_clear, dim3(grid_for(n, 256)), dim3(256), 0, stream, arrive, n_arrive, count,
                       n_count, slots, n_slot_values);
    return hipGetLastError();
}

hipError_t launch_cc_cost(const CollTable &t, const echo_cc_table *tables, const echo_scenario *scen,
                          int32_t n_scen, int64_t *cost, unsigned *status, hipStream_t stream) {
    if (t.n == 0 || n_scen == 0) return hipSuccess;
    // one lane per (collective, scenario): collectives along x, 64-scenario tiles along y
    const unsigned tiles = (unsigned)std::min<int64_t>((n_scen + 63) / 64, 65535);
    hipLaunchKernelGGL(k_cc_cost, dim3((unsigned)t.n, tiles), dim3(64), 0, stream, t, tables, scen, n_scen, cost,
                       status);
    return hipGetLastError();
}

hipError_t launch_walk(const WalkArgs &a, int32_t n_blocks, hipStream_t stream) {
    WalkArgs args = a;
    void *params[] = {&args};
    const WalkKernel k = walk_kernel(walk_input(a.tmask != nullptr || a.ext != nullptr, a.ext != nullptr,
                                                a.flag_rows != 0),
                                     a.final_pass != 0, a.digest != nullptr);
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k), dim3((unsigned)(n_blocks * a.tiles)),
                                      dim3(kBlockWalkers * kLanes), params, 0, stream);
}

template <bool PRORATE, bool DETECT, int FOREST, int NC>
void launch_overlap_kernel(const OverlapArgs &a, dim3 grid, dim3 block, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((k_overlap<PRORATE, DETECT, FOREST, NC>), grid, block, lds, stream, a);
}

template <int NC>
hipError_t launch_overlap_nc(const OverlapArgs &a, int32_t n_ranks, hipStream_t stream) {
    const int64_t units = (int64_t)n_ranks * a.n_tiles;
    const dim3 grid((unsigned)units), block(kLanes);
    // a.ext: extra-time output (prorating and/or ensemble factors); a.forest_nodes: ensemble
    const bool forest = a.forest_nodes != nullptr, prorate = a.prorate != 0;
    if (forest && a.fx.n_words > 0) {
        // compact ensemble in LDS: kFxWaves (rank, tile) units per workgroup share its nodes
        const dim3 g2((unsigned)((units + kFxWaves - 1) / kFxWaves)), b2(kLanes * kFxWaves);
        const size_t lds = sizeof(uint32_t) * ((size_t)a.fx.n_words + (size_t)a.n_trees);
        if (prorate && a.chg) launch_overlap_kernel<true, true, 2, NC>(a, g2, b2, lds, stream);
        else if (prorate) launch_overlap_kernel<true, false, 2, NC>(a, g2, b2, lds, stream);
        else if (a.chg) launch_overlap_kernel<false, true, 2, NC>(a, g2, b2, lds, stream);
        else launch_overlap_kernel<false, false, 2, NC>(a, g2, b2, lds, stream);
    } else if (forest) {
        if (prorate && a.chg) launch_overlap_kernel<true, true, 1, NC>(a, grid, block, 0, stream);
        else if (prorate) launch_overlap_kernel<true, false, 1, NC>(a, grid, block, 0, stream);
        else if (a.chg) launch_overlap_kernel<false, true, 1, NC>(a, grid, block, 0, stream);
        else launch_overlap_kernel<false, false, 1, NC>(a, grid, block, 0, stream);
    } else if (prorate && a.chg) launch_overlap_kernel<true, true, 0, NC>(a, grid, block, 0, stream);
    else if (prorate) launch_overlap_kernel<true, false, 0, NC>(a, grid, block, 0, stream);
    else if (a.chg) launch_overlap_kernel<false, true, 0, NC>(a, grid, block, 0, stream);
    else launch_overlap_kernel<false, false, 0, NC>(a, grid, block, 0, stream);
    return hipGetLastError();
}

hipError_t launch_overlap(const OverlapArgs &a, int32_t n_ranks, hipStream_t stream) {
    if (a.max_comm_streams > 4) return launch_overlap_nc<kStreams>(a, n_ranks, stream);
    return launch_overlap_nc<4>(a, n_ranks, stream);
}

hipError_t launch_forest_bins(const DeviceGraph &g, int64_t n_cp, const CompactForest &fx, hipStream_t stream) {
    const int64_t n = std::max<int64_t>(g.colls.n, n_cp);
    hipLaunchKernelGGL(k_forest_bins, dim3(grid_for(n, 256)), dim3(256), 0, stream, g.colls, g.cp, n_cp, fx);
    return hipGetLastError();
}

hipError_t launch_settle(unsigned *chg, int32_t n_scen, int32_t *refinements, unsigned *stable,
                         hipStream_t stream) {
    hipLaunchKernelGGL(k_settle, dim3(1), dim3(256), 0, stream, chg, n_scen, refinements, stable);
    return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256)), dim3(256), 0, stream, p, n, v);
    return hipGetLastError();
}

// Workspace of echo_compose_batch_static: one fixed array in every GPU's copy of the
// code object, held from the code object's load until the process ends.  In host code
// `scratch` names a host-side stand-in only; kernels get the device address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[ECHO_SCRATCH_BYTES];

hipError_t scratch_buffer(int device, void **ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    *ptr = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        // the caller has made `device` current: its copy of the array
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[device] = p;
    }
    *ptr = addr[device];
    return hipSuccess;
}

hipError_t walk_capacity(int device, int64_t workgroups[kWalkVariants]) {
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    for (int v = 0; v < kWalkVariants; ++v) {
        int per_cu = 0;
        const WalkKernel k = walk_kernel(v & 3, v & 4, v & 8);
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(k),
                                                         kBlockWalkers * kLanes, 0);
        if (e != hipSuccess) return e;
        workgroups[v] = (int64_t)per_cu * cus;
    }
    return hipSuccess;
}

}  // namespace echo
