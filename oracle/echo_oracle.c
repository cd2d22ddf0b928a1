/*
 * echo_oracle.c -- plain CPU reference of Echo's timeline composer.
 *
 * TEST INFRASTRUCTURE.  This file is the oracle that the HIP implementation is
 * checked against.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it.  It shares no code, header or table with
 * the HIP library; both read the same seeded input arrays and nothing else.
 *
 * What it computes, in the paper's order (Echo, arXiv 2412.12487):
 *   1. CC estimator (Sec. 5.3, Eq. 1-5, chunk sizes of Table 6): the running
 *      time T(c) of every collective for one scenario.
 *   2. Timeline composer (Sec. 4.2): an event-driven replay that takes every
 *      operator off a time-ordered event queue and puts it on its rank's
 *      stream timelines.  A collective kernel first synchronises -- it waits
 *      until every member of its group has launched, the last launch fixes
 *      the start -- and then executes for T(c) (Sec. 5.2).  P2P send/recv is
 *      a two-member group.
 *   3. Validator (Sec. 6 and the slowdown definition next to Table 2): every
 *      computation operator that overlaps a communication operator of the
 *      same rank has its duration multiplied by the slowdown factor (ratio of
 *      running time with overlap to running time without), and the timeline
 *      is composed again.
 *
 * Readings taken where the paper is silent:
 *   - stream timelines are FIFO in program order; the k-th op of a stream
 *     waits for the (k-1)-th to finish;
 *   - a comm op starts at its own launch and finishes at barrier + T(c);
 *   - the untyped (N-1) term of Eq. 3 and Eq. 4 is multiplied by beta;
 *   - eta = ceil(S / (N * chunk)) for ring kernels, ceil(S / chunk) for tree
 *     and P2P; gamma is replaced by beta when all members share a server;
 *   - log2(M) is the ceiling log2 (binary-tree depth);
 *   - beta, gamma and the reduce time come from the scenario's bandwidths
 *     with ceiling division;
 *   - overlap is same-rank, computation op vs any comm op, intervals [s, f)
 *     with a non-empty intersection; several overlaps take the largest
 *     factor; memcpy and comm durations are never inflated; R refinements
 *     each recompose from the un-inflated durations.
 *
 * All times are int64 nanoseconds; slowdown factors are Q16 fixed point.
 * Every value this file produces is exact integer arithmetic.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

enum { OK = 0, E_ARG = -1, E_RANGE = -2, E_MATCH = -3, E_CYCLE = -4, E_NOMEM = -5 };
enum { COMPUTE = 0, COMM = 1, MEMCPY = 2 };
enum { AR = 0, AG = 1, RS = 2, P2P = 3 };
enum { RING = 0, TREE = 1 };

#define NSTREAM 8
#define NCLASS 8
#define TIME_LIMIT ((int64_t)1 << 62)
#define DUR_LIMIT ((int64_t)1 << 43)
#define BYTES_LIMIT ((int64_t)1 << 50)
#define KNOB_LIMIT ((int64_t)1 << 40)
#define Q16_ONE 65536u

typedef unsigned __int128 u128;

/* ------------------------------------------------------------------ */
/* Inputs                                                              */
/* ------------------------------------------------------------------ */
typedef struct {
    int64_t n_ops;
    int32_t n_ranks, gpus_per_node;
    const int32_t *op_rank;
    const uint8_t *op_stream, *op_kind, *op_class;
    const int64_t *op_dur, *op_coll, *pred_off;
    const int32_t *pred_idx;
    int64_t n_colls;
    const uint8_t *coll_type;
    const int64_t *coll_bytes;
    /* optional membership each collective is costed with (Sec. 8.5, DDP mode: one
       DP replica simulated alone, its collectives keeping their whole group's size) */
    const int32_t *coll_N, *coll_M, *coll_K;
} graph_t;

/* A CC parameter table (Sec. 5.3 offline profiling; rows like Table 6): per
   row, the largest message it serves, chunk size, alpha, per-chunk beta and
   gamma (ns) and reduce throughput (MB/s). */
#define CC_ROWS 7
typedef struct {
    int64_t max_bytes[CC_ROWS], chunk[CC_ROWS], alpha[CC_ROWS], beta[CC_ROWS], gamma[CC_ROWS],
        reduce[CC_ROWS];
} cc_table_t;

/* A gradient-boosted tree ensemble predicting the slowdown factor (Sec. 6,
   features after Table 4, trees of depth <= 12 after Table 5).  Node: feature
   index (-1: leaf), children, leaf value (Q16 contribution), threshold (go
   left when x[feature] < threshold). */
#define NFEAT 12
#define NMETRIC 4
#define TREE_DEPTH 12
typedef struct {
    int32_t feature, left, right, value;
    int64_t threshold;
} tree_node_t;
typedef struct {
    const tree_node_t *nodes;
    int64_t n_nodes;
    const int32_t *roots;
    int32_t n_trees;
    int32_t base;                    /* base score (Q16) */
    const int64_t *class_metrics;    /* [8 classes][NMETRIC] kernel metrics, features 8..11 */
} forest_t;

typedef struct {
    int64_t alpha, bw_intra, bw_inter, reduce;
    uint64_t jseed;
    uint32_t jstream;
    int32_t jamp;
    uint8_t algo;
    uint8_t cc_model;        /* 0: Eq. 2-5; 1: alpha-beta baseline */
    const cc_table_t *table; /* parameters of Eq. 2-5 from this table, or NULL: from bandwidths */
    const uint32_t *slow;    /* [8 classes][4 collective types] */
    const forest_t *forest;  /* factors predicted by this ensemble instead of taken from slow */
} scen_t;

/* Structure derived once from the graph and shared by all scenarios. */
typedef struct {
    int64_t *npred;          /* distinct predecessors of each op                 */
    int64_t *succ_off;       /* successors (CSR)                                 */
    int64_t *succ;
    int64_t *mem_off;        /* members of each collective (CSR), program order  */
    int64_t *mem;
    int64_t *cN;             /* member ops present: the arrivals that complete a barrier */
    int64_t *cM, *cK;        /* distinct servers, max members per server (of those present) */
    int64_t *tN, *tM, *tK;   /* N, M, K the cost formulas use (given, else cN, cM, cK) */
    int64_t *cl_off;         /* comm ops of each (rank, stream), program order   */
    int64_t *cl;
} derived_t;

static void set_err(char *err, int64_t len, const char *msg, long long a, long long b) {
    if (err && len > 0) snprintf(err, (size_t)len, msg, a, b);
}

/* ------------------------------------------------------------------ */
/* Sec. 5.3: white-box CC execution model                              */
/* ------------------------------------------------------------------ */

/* Table 6: NCCL chunk size for a tensor size (MB read as MiB, chunk as 10^3 B). */
static int64_t chunk_bytes(int64_t S) {
    const int64_t MiB = 1024 * 1024;
    if (S <= 4 * MiB) return 18000;
    if (S <= 8 * MiB) return 36000;
    if (S <= 16 * MiB) return 72000;
    if (S <= 32 * MiB) return 72000;
    if (S <= 64 * MiB) return 72000;
    if (S <= 128 * MiB) return 144000;
    return 288000;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int64_t ceil_log2(int64_t x) {
    int64_t k = 0;
    while (((int64_t)1 << k) < x) k++;
    return k;
}

/* Eq. 2 (ring all-gather), Eq. 3 (ring reduce-scatter), Eq. 4 (ring
 * all-reduce), Eq. 5 (tree all-reduce) and point-to-point as one chunked hop.
 * Returns -1 when the exact result is >= 2^62. */
/* Alpha-beta baseline (not the paper's model; a what-if reference): the
 * latency-bandwidth cost of the ring and binomial-tree algorithms after Thakur,
 * Rabenseifner and Gropp (IJHPCA 2005), rounding each step up to a nanosecond.
 * Ring steps move one N-th of the message, tree steps all of it. */
static int64_t cc_time_alpha_beta(int type, int64_t S, int64_t N, int64_t M, const scen_t *sc) {
    const int64_t B = M > 1 ? sc->bw_inter : sc->bw_intra;
    const int64_t part = ceil_div(S, N);
    const u128 alpha = (u128)sc->alpha, n1 = (u128)(N - 1);
    const u128 t_part = (u128)ceil_div(part * 1000, B), r_part = (u128)ceil_div(part * 1000, sc->reduce);
    const u128 t_all = (u128)ceil_div(S * 1000, B), r_all = (u128)ceil_div(S * 1000, sc->reduce);
    u128 T;
    switch (type) {
    case AG: T = n1 * (alpha + t_part); break;                         /* N-1 steps */
    case RS: T = n1 * (alpha + t_part + r_part); break;                /* N-1 steps, each reduces */
    case AR:
        if (sc->algo == TREE) T = (u128)ceil_log2(N) * (2 * alpha + 2 * t_all + r_all);  /* reduce + broadcast */
        else T = n1 * (2 * alpha + 2 * t_part + r_part);              /* reduce-scatter + all-gather */
        break;
    default: T = alpha + t_all; break;                                 /* one hop */
    }
    if (T >= (u128)TIME_LIMIT) return -1;
    return (int64_t)T;
}

static int64_t cc_time(int type, int64_t S, int64_t N, int64_t M, int64_t K, const scen_t *sc) {
    if (sc->cc_model == 1) return cc_time_alpha_beta(type, S, N, M, sc);
    int64_t chunk, a, b, c, red;
    if (sc->table) {
        /* the first row whose bound covers S; the last row takes every larger S */
        int i = 0;
        while (i < CC_ROWS - 1 && S > sc->table->max_bytes[i]) i++;
        chunk = sc->table->chunk[i];
        a = sc->table->alpha[i];
        b = sc->table->beta[i];
        c = sc->table->gamma[i];
        red = sc->table->reduce[i];
    } else {
        chunk = chunk_bytes(S);
        a = sc->alpha;
        b = ceil_div(chunk * 1000, sc->bw_intra);   /* intra-server per chunk */
        c = ceil_div(chunk * 1000, sc->bw_inter);   /* inter-server per chunk */
        red = sc->reduce;
    }
    const u128 alpha = (u128)a;
    const u128 beta = (u128)b;
    const u128 g = M > 1 ? (u128)c : beta;                           /* slowest hop in the group */
    const u128 eta_ring = (u128)ceil_div(S, N * chunk);              /* ring rounds */
    const u128 eta_chunks = (u128)ceil_div(S, chunk);                /* pipelined chunks */
    const u128 reduce = (u128)ceil_div(S * 1000, red);               /* delta * tensor_size */
    const u128 n1 = (u128)(N - 1);
    u128 T;
    switch (type) {
    case AG:
        T = alpha + g * eta_ring * n1;
        break;
    case RS:
        T = alpha + eta_ring * (n1 * beta + n1 * g) + reduce;
        break;
    case AR:
        if (sc->algo == TREE)
            T = alpha + g * (eta_chunks > 0 ? eta_chunks - 1 : 0) + 2 * beta * (u128)(K - 1)
                + 2 * g * (u128)ceil_log2(M) + reduce;
        else
            T = alpha + eta_ring * (n1 * beta + 2 * n1 * g) + reduce;
        break;
    default: /* P2P */
        T = alpha + eta_chunks * g;
        break;
    }
    if (T >= (u128)TIME_LIMIT) return -1;
    return (int64_t)T;
}

/* ------------------------------------------------------------------ */
/* Scenario expansion: jittered base durations                          */
/* ------------------------------------------------------------------ */

/* k-th output (k >= 1) of SplitMix64 (Steele, Lea, Flood, OOPSLA 2014) seeded with `seed`. */
static uint64_t splitmix64_at(uint64_t seed, uint64_t k) {
    uint64_t z = seed + k * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Q16 scaling with round-half-up: d * f / 65536. */
static int64_t q16_scale(int64_t d, uint64_t f) {
    return (int64_t)(((uint64_t)d * f + 32768u) >> 16);
}

/* D(v): base duration with the scenario's uniform jitter of amplitude A (Q16). */
static int64_t base_duration(const graph_t *g, const scen_t *sc, int64_t v) {
    const int64_t d0 = g->op_dur[v];
    if (sc->jamp == 0) return d0;
    const uint64_t k = ((uint64_t)sc->jstream << 36) + (uint64_t)v + 1;
    const uint64_t u = splitmix64_at(sc->jseed, k);
    const int64_t A = sc->jamp;
    const int64_t J = (int64_t)(((u >> 32) * (uint64_t)(2 * A + 1)) >> 32) - A;
    return q16_scale(d0, (uint64_t)(Q16_ONE + J));
}

/* Mixing function of the timeline digest: the SplitMix64 output function. */
static uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* ------------------------------------------------------------------ */
/* Sec. 4.2: event-driven timeline composer                             */
/* ------------------------------------------------------------------ */
typedef struct { int64_t t, v; } event_t;

typedef struct {
    event_t *a;
    int64_t n;
} heap_t;

static int ev_less(event_t x, event_t y) { return x.t < y.t || (x.t == y.t && x.v < y.v); }

static void heap_push(heap_t *h, event_t e) {
    int64_t i = h->n++;
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (!ev_less(e, h->a[p])) break;
        h->a[i] = h->a[p];
        i = p;
    }
    h->a[i] = e;
}

static event_t heap_pop(heap_t *h) {
    event_t top = h->a[0], last = h->a[--h->n];
    int64_t i = 0;
    for (;;) {
        int64_t c = 2 * i + 1;
        if (c >= h->n) break;
        if (c + 1 < h->n && ev_less(h->a[c + 1], h->a[c])) c++;
        if (!ev_less(h->a[c], last)) break;
        h->a[i] = h->a[c];
        i = c;
    }
    if (h->n > 0) h->a[i] = last;
    return top;
}

typedef struct {
    int64_t *pending, *ready, *arrived, *barrier, *dur;
    heap_t heap;
} work_t;

/* One replay of the whole job with per-op durations dur[] and collective
 * times cost[]; fills s[] (launch on the stream) and f[] (finish). */
static int compose(const graph_t *g, const derived_t *dv, const int64_t *dur, const int64_t *cost,
                   int64_t *s, int64_t *f, work_t *w, char *err, int64_t errlen) {
    const int64_t n = g->n_ops;
    for (int64_t v = 0; v < n; v++) {
        w->pending[v] = dv->npred[v];
        w->ready[v] = 0;
    }
    for (int64_t c = 0; c < g->n_colls; c++) {
        w->arrived[c] = 0;
        w->barrier[c] = 0;
    }
    w->heap.n = 0;

    /* Launch op v at time t: compute/memcpy run for their duration; a comm
     * op registers its arrival and, once the last member of its group has
     * launched, every member finishes at barrier + T(c). */
    int64_t finished = 0;
#define LAUNCH(vv, tt)                                                              \
    do {                                                                            \
        const int64_t v_ = (vv), t_ = (tt);                                         \
        s[v_] = t_;                                                                 \
        if (g->op_kind[v_] == COMM) {                                               \
            const int64_t c_ = g->op_coll[v_];                                      \
            w->arrived[c_]++;                                                       \
            if (t_ > w->barrier[c_]) w->barrier[c_] = t_;                           \
            if (w->arrived[c_] == dv->cN[c_]) {                                     \
                const int64_t fin_ = w->barrier[c_] + cost[c_];                     \
                if (fin_ >= TIME_LIMIT) goto overflow;                              \
                for (int64_t j_ = dv->mem_off[c_]; j_ < dv->mem_off[c_ + 1]; j_++) { \
                    f[dv->mem[j_]] = fin_;                                          \
                    heap_push(&w->heap, (event_t){fin_, dv->mem[j_]});             \
                }                                                                   \
            }                                                                       \
        } else {                                                                    \
            const int64_t fin_ = t_ + dur[v_];                                      \
            if (fin_ >= TIME_LIMIT) goto overflow;                                  \
            f[v_] = fin_;                                                           \
            heap_push(&w->heap, (event_t){fin_, v_});                              \
        }                                                                           \
    } while (0)

    for (int64_t v = 0; v < n; v++)
        if (w->pending[v] == 0) LAUNCH(v, 0);
    while (w->heap.n > 0) {
        const event_t e = heap_pop(&w->heap);
        finished++;
        for (int64_t j = dv->succ_off[e.v]; j < dv->succ_off[e.v + 1]; j++) {
            const int64_t u = dv->succ[j];
            if (e.t > w->ready[u]) w->ready[u] = e.t;
            if (--w->pending[u] == 0) LAUNCH(u, w->ready[u]);
        }
    }
#undef LAUNCH
    if (finished != n) {
        for (int64_t c = 0; c < g->n_colls; c++)
            if (w->arrived[c] < dv->cN[c] && w->arrived[c] > 0) {
                set_err(err, errlen, "deadlock: collective %lld has %lld members launched",
                        (long long)c, (long long)w->arrived[c]);
                return E_CYCLE;
            }
        set_err(err, errlen, "deadlock: %lld of %lld ops never ran", (long long)(n - finished),
                (long long)n);
        return E_CYCLE;
    }
    return OK;
overflow:
    set_err(err, errlen, "a finish time reached 2^62 ns", 0, 0);
    return E_RANGE;
}

/* ------------------------------------------------------------------ */
/* Sec. 6: overlap with communication -> slowdown factor per compute op */
/* ------------------------------------------------------------------ */
/* Factor predicted for a compute op from feature vector x: the base score plus one
 * leaf value per tree, kept inside the factor range [65536, 2^20). */
static uint32_t forest_predict(const forest_t *fo, const int64_t *x) {
    int64_t sum = fo->base;
    for (int32_t t = 0; t < fo->n_trees; t++) {
        int32_t i = fo->roots[t];
        while (fo->nodes[i].feature >= 0)
            i = x[fo->nodes[i].feature] < fo->nodes[i].threshold ? fo->nodes[i].left : fo->nodes[i].right;
        sum += fo->nodes[i].value;
    }
    if (sum < Q16_ONE) sum = Q16_ONE;
    if (sum >= (1 << 20)) sum = (1 << 20) - 1;
    return (uint32_t)sum;
}

/* Features of compute op v overlapped by comm ops of collective type t (after
 * Table 4): kernel class, profiled running time (base duration, no jitter),
 * collective type, largest message ("bucket size") and most members among the
 * overlapping comm ops of that type, the scenario's all-reduce algorithm and
 * bandwidths, and four per-class kernel metrics. */
static void forest_features(const graph_t *g, const scen_t *sc, int64_t v, int t, int64_t smax, int64_t nmax,
                            int64_t *x) {
    const int cls = g->op_class[v];
    x[0] = cls;
    x[1] = g->op_dur[v];
    x[2] = t;
    x[3] = smax;
    x[4] = nmax;
    x[5] = sc->algo;
    x[6] = sc->bw_intra;
    x[7] = sc->bw_inter;
    for (int k = 0; k < NMETRIC; k++) x[8 + k] = sc->forest->class_metrics[cls * NMETRIC + k];
}

static void overlap_factors(const graph_t *g, const derived_t *dv, const scen_t *sc,
                            const int64_t *s, const int64_t *f, uint32_t *F, int64_t *O, int64_t *lo_buf,
                            int64_t *hi_buf) {
    for (int64_t v = 0; v < g->n_ops; v++) {
        F[v] = Q16_ONE;
        O[v] = 0;
        if (g->op_kind[v] != COMPUTE) continue;
        const int64_t r = g->op_rank[v], sv = s[v], fv = f[v];
        const uint32_t *row = sc->slow + 4 * g->op_class[v];
        uint32_t best = Q16_ONE;
        int64_t n_iv = 0;           /* overlapping comm intervals, clipped to [sv, fv) */
        int64_t smax[4] = {-1, -1, -1, -1}, nmax[4] = {0, 0, 0, 0};   /* per type, for the forest */
        for (int k = 0; k < NSTREAM; k++) {
            const int64_t lo0 = dv->cl_off[r * NSTREAM + k], hi0 = dv->cl_off[r * NSTREAM + k + 1];
            /* Comm ops of one stream are FIFO, so their finish times are sorted:
             * binary search the first one that ends after v starts. */
            int64_t lo = lo0, hi = hi0;
            while (lo < hi) {
                const int64_t mid = lo + (hi - lo) / 2;
                if (f[dv->cl[mid]] > sv) hi = mid; else lo = mid + 1;
            }
            for (int64_t j = lo; j < hi0; j++) {
                const int64_t c = dv->cl[j];
                if (s[c] >= fv) break;
                const int64_t a = sv > s[c] ? sv : s[c], b = fv < f[c] ? fv : f[c];
                if (a < b) {
                    const int64_t cc = g->op_coll[c];
                    const int ty = g->coll_type[cc];
                    const uint32_t x = row[ty];
                    if (x > best) best = x;
                    if (g->coll_bytes[cc] > smax[ty]) smax[ty] = g->coll_bytes[cc];
                    if (dv->tN[cc] > nmax[ty]) nmax[ty] = dv->tN[cc];
                    lo_buf[n_iv] = a;
                    hi_buf[n_iv] = b;
                    n_iv++;
                }
            }
        }
        if (sc->forest) {
            /* the ensemble's prediction for each overlapping collective type; the largest counts */
            best = Q16_ONE;
            for (int ty = 0; ty < 4; ty++) {
                if (smax[ty] < 0) continue;
                int64_t x[NFEAT];
                forest_features(g, sc, v, ty, smax[ty], nmax[ty], x);
                const uint32_t p = forest_predict(sc->forest, x);
                if (p > best) best = p;
            }
        }
        F[v] = best;
        /* length of the union of the clipped intervals: sort by start, then sweep */
        for (int64_t i = 1; i < n_iv; i++) {
            const int64_t a = lo_buf[i], b = hi_buf[i];
            int64_t j = i - 1;
            while (j >= 0 && lo_buf[j] > a) {
                lo_buf[j + 1] = lo_buf[j];
                hi_buf[j + 1] = hi_buf[j];
                j--;
            }
            lo_buf[j + 1] = a;
            hi_buf[j + 1] = b;
        }
        int64_t covered = 0, end = sv;
        for (int64_t i = 0; i < n_iv; i++) {
            const int64_t a = lo_buf[i] > end ? lo_buf[i] : end;
            if (hi_buf[i] > a) {
                covered += hi_buf[i] - a;
                end = hi_buf[i];
            }
        }
        O[v] = covered;
    }
}

/* Duration of compute op v in a refined pass (Sec. 6): the whole base duration
 * D runs F times slower; prorated, only the overlapped part does -- the
 * overlapped length measured on the previous timeline, capped at D. */
static int64_t inflated(int64_t D, uint32_t F, int64_t overlapped, int prorate) {
    if (!prorate) return q16_scale(D, F);
    const int64_t o = overlapped < D ? overlapped : D;
    return D - o + q16_scale(o, F);
}

/* ------------------------------------------------------------------ */
/* Validation of the graph and the derived structure                    */
/* ------------------------------------------------------------------ */
static int check_graph(const graph_t *g, char *err, int64_t errlen) {
    if (g->n_ops < 0 || g->n_ranks < 1 || g->gpus_per_node < 1 || g->n_colls < 0) {
        set_err(err, errlen, "bad sizes (n_ops %lld, n_colls %lld)", (long long)g->n_ops,
                (long long)g->n_colls);
        return E_ARG;
    }
    if (g->n_ops >= ((int64_t)1 << 31)) {
        set_err(err, errlen, "too many ops: %lld", (long long)g->n_ops, 0);
        return E_RANGE;
    }
    if (g->pred_off[0] != 0) {
        set_err(err, errlen, "pred_off[0] = %lld", (long long)g->pred_off[0], 0);
        return E_ARG;
    }
    for (int64_t v = 0; v < g->n_ops; v++) {
        const int32_t r = g->op_rank[v];
        if (r < 0 || r >= g->n_ranks || (v > 0 && r < g->op_rank[v - 1]) || g->op_stream[v] >= NSTREAM
            || g->op_kind[v] > MEMCPY || g->op_class[v] >= NCLASS) {
            set_err(err, errlen, "op %lld has a bad rank/stream/kind/class", (long long)v, 0);
            return E_ARG;
        }
        if (g->op_kind[v] == COMM) {
            if (g->op_coll[v] < 0 || g->op_coll[v] >= g->n_colls) {
                set_err(err, errlen, "comm op %lld has collective %lld", (long long)v,
                        (long long)g->op_coll[v]);
                return E_ARG;
            }
        } else {
            if (g->op_coll[v] != -1) {
                set_err(err, errlen, "non-comm op %lld names collective %lld", (long long)v,
                        (long long)g->op_coll[v]);
                return E_ARG;
            }
            if (g->op_dur[v] < 0 || g->op_dur[v] >= DUR_LIMIT) {
                set_err(err, errlen, "op %lld duration %lld out of range", (long long)v,
                        (long long)g->op_dur[v]);
                return E_RANGE;
            }
        }
        if (g->pred_off[v + 1] < g->pred_off[v]) {
            set_err(err, errlen, "pred_off decreases at op %lld", (long long)v, 0);
            return E_ARG;
        }
        for (int64_t j = g->pred_off[v]; j < g->pred_off[v + 1]; j++) {
            const int64_t u = g->pred_idx[j];
            if (u < 0 || u >= v || g->op_rank[u] != r) {
                set_err(err, errlen, "op %lld depends on op %lld (must be an earlier op of its rank)",
                        (long long)v, (long long)u);
                return E_ARG;
            }
        }
    }
    for (int64_t c = 0; c < g->n_colls; c++) {
        if (g->coll_type[c] > P2P) {
            set_err(err, errlen, "collective %lld has type %lld", (long long)c, (long long)g->coll_type[c]);
            return E_ARG;
        }
        if (g->coll_bytes[c] < 0 || g->coll_bytes[c] >= BYTES_LIMIT) {
            set_err(err, errlen, "collective %lld size %lld out of range", (long long)c,
                    (long long)g->coll_bytes[c]);
            return E_RANGE;
        }
    }
    return OK;
}

static int check_scen(const scen_t *sc, char *err, int64_t errlen) {
    if (sc->alpha < 0 || sc->alpha >= KNOB_LIMIT || sc->bw_intra < 1 || sc->bw_intra >= KNOB_LIMIT
        || sc->bw_inter < 1 || sc->bw_inter >= KNOB_LIMIT || sc->reduce < 1 || sc->reduce >= KNOB_LIMIT
        || sc->jamp < 0 || sc->jamp > 65535 || sc->algo > TREE || sc->cc_model > 1) {
        set_err(err, errlen, "scenario knob out of range", 0, 0);
        return E_RANGE;
    }
    for (int i = 0; i < NCLASS * 4; i++)
        if (sc->slow[i] < Q16_ONE || sc->slow[i] >= (1u << 20)) {
            set_err(err, errlen, "slowdown entry %lld = %lld out of range", (long long)i, (long long)sc->slow[i]);
            return E_RANGE;
        }
    return OK;
}

static void free_derived(derived_t *d) {
    free(d->npred); free(d->succ_off); free(d->succ); free(d->mem_off); free(d->mem);
    free(d->cN); free(d->cM); free(d->cK); free(d->tN); free(d->tM); free(d->tK); free(d->cl_off); free(d->cl);
}

static int cmp_i64(const void *a, const void *b) {
    const int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

/* Predecessors of v: the previous op on its stream plus its explicit
 * dependencies, without repeats.  Written into buf (sorted); returns count. */
static int64_t preds_of(const graph_t *g, const int64_t *stream_prev, int64_t v, int64_t *buf) {
    int64_t k = 0;
    if (stream_prev[v] >= 0) buf[k++] = stream_prev[v];
    for (int64_t j = g->pred_off[v]; j < g->pred_off[v + 1]; j++) buf[k++] = g->pred_idx[j];
    qsort(buf, (size_t)k, sizeof(int64_t), cmp_i64);
    int64_t m = 0;
    for (int64_t i = 0; i < k; i++)
        if (m == 0 || buf[i] != buf[m - 1]) buf[m++] = buf[i];
    return m;
}

static int derive(const graph_t *g, derived_t *d, char *err, int64_t errlen) {
    const int64_t n = g->n_ops, nc = g->n_colls, R = g->n_ranks;
    memset(d, 0, sizeof(*d));
    int64_t *stream_prev = malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *last = malloc(sizeof(int64_t) * (size_t)R * NSTREAM);
    int64_t maxp = 1;
    for (int64_t v = 0; v < n; v++)
        if (g->pred_off[v + 1] - g->pred_off[v] + 1 > maxp) maxp = g->pred_off[v + 1] - g->pred_off[v] + 1;
    int64_t *buf = malloc(sizeof(int64_t) * (size_t)maxp);
    d->npred = calloc((size_t)n + 1, sizeof(int64_t));
    d->succ_off = calloc((size_t)n + 2, sizeof(int64_t));
    d->mem_off = calloc((size_t)nc + 2, sizeof(int64_t));
    d->cN = calloc((size_t)nc + 1, sizeof(int64_t));
    d->cM = calloc((size_t)nc + 1, sizeof(int64_t));
    d->cK = calloc((size_t)nc + 1, sizeof(int64_t));
    d->tN = calloc((size_t)nc + 1, sizeof(int64_t));
    d->tM = calloc((size_t)nc + 1, sizeof(int64_t));
    d->tK = calloc((size_t)nc + 1, sizeof(int64_t));
    d->cl_off = calloc((size_t)R * NSTREAM + 2, sizeof(int64_t));
    if (!stream_prev || !last || !buf || !d->npred || !d->succ_off || !d->mem_off || !d->cN || !d->cM
        || !d->cK || !d->tN || !d->tM || !d->tK || !d->cl_off) goto nomem;
    for (int64_t i = 0; i < R * NSTREAM; i++) last[i] = -1;
    for (int64_t v = 0; v < n; v++) {
        const int64_t key = (int64_t)g->op_rank[v] * NSTREAM + g->op_stream[v];
        stream_prev[v] = last[key];
        last[key] = v;
    }
    /* successor CSR */
    for (int64_t v = 0; v < n; v++) {
        const int64_t m = preds_of(g, stream_prev, v, buf);
        d->npred[v] = m;
        for (int64_t i = 0; i < m; i++) d->succ_off[buf[i] + 1]++;
    }
    for (int64_t v = 0; v < n; v++) d->succ_off[v + 1] += d->succ_off[v];
    d->succ = malloc(sizeof(int64_t) * (size_t)(d->succ_off[n] + 1));
    int64_t *fill = malloc(sizeof(int64_t) * (size_t)(n + 1));
    if (!d->succ || !fill) { free(fill); goto nomem; }
    memcpy(fill, d->succ_off, sizeof(int64_t) * (size_t)n);
    for (int64_t v = 0; v < n; v++) {
        const int64_t m = preds_of(g, stream_prev, v, buf);
        for (int64_t i = 0; i < m; i++) d->succ[fill[buf[i]]++] = v;
    }
    free(fill);
    /* members of each collective; N, M (servers), K (max members per server) */
    for (int64_t v = 0; v < n; v++)
        if (g->op_kind[v] == COMM) d->mem_off[g->op_coll[v] + 1]++;
    for (int64_t c = 0; c < nc; c++) {
        d->cN[c] = d->mem_off[c + 1];
        if (d->cN[c] == 0) {
            set_err(err, errlen, "collective %lld has no member op", (long long)c, 0);
            free(stream_prev); free(last); free(buf); free_derived(d);
            return E_MATCH;
        }
        d->mem_off[c + 1] += d->mem_off[c];
    }
    d->mem = malloc(sizeof(int64_t) * (size_t)(d->mem_off[nc] + 1));
    fill = malloc(sizeof(int64_t) * (size_t)(nc + 1));
    if (!d->mem || !fill) { free(fill); goto nomem; }
    memcpy(fill, d->mem_off, sizeof(int64_t) * (size_t)nc);
    for (int64_t v = 0; v < n; v++)
        if (g->op_kind[v] == COMM) d->mem[fill[g->op_coll[v]]++] = v;
    free(fill);
    for (int64_t c = 0; c < nc; c++) {
        /* members are in ascending op id, hence ascending rank and server */
        int64_t servers = 0, best = 0, run = 0, prev_node = -1;
        for (int64_t j = d->mem_off[c]; j < d->mem_off[c + 1]; j++) {
            const int64_t node = g->op_rank[d->mem[j]] / g->gpus_per_node;
            if (node != prev_node) { servers++; run = 0; prev_node = node; }
            run++;
            if (run > best) best = run;
        }
        d->cM[c] = servers;
        d->cK[c] = best;
        if (g->coll_type[c] == P2P && d->cN[c] != 2) {
            set_err(err, errlen, "P2P collective %lld has %lld members", (long long)c, (long long)d->cN[c]);
            free(stream_prev); free(last); free(buf); free_derived(d);
            return E_MATCH;
        }
        d->tN[c] = d->cN[c];
        d->tM[c] = d->cM[c];
        d->tK[c] = d->cK[c];
        if (g->coll_N) {
            /* the whole group: at least the members present, M servers of at most K each */
            const int64_t N = g->coll_N[c], M = g->coll_M[c], K = g->coll_K[c];
            if (N < d->cN[c] || M < 1 || M > N || K < 1 || K > N || M * K < N
                || (g->coll_type[c] == P2P && N != 2)) {
                set_err(err, errlen, "collective %lld: given membership inconsistent (N %lld)", (long long)c,
                        (long long)N);
                free(stream_prev); free(last); free(buf); free_derived(d);
                return E_ARG;
            }
            d->tN[c] = N;
            d->tM[c] = M;
            d->tK[c] = K;
        }
    }
    /* comm ops per (rank, stream), program order */
    for (int64_t v = 0; v < n; v++)
        if (g->op_kind[v] == COMM) d->cl_off[(int64_t)g->op_rank[v] * NSTREAM + g->op_stream[v] + 1]++;
    for (int64_t i = 0; i < R * NSTREAM; i++) d->cl_off[i + 1] += d->cl_off[i];
    d->cl = malloc(sizeof(int64_t) * (size_t)(d->cl_off[R * NSTREAM] + 1));
    fill = malloc(sizeof(int64_t) * (size_t)(R * NSTREAM + 1));
    if (!d->cl || !fill) { free(fill); goto nomem; }
    memcpy(fill, d->cl_off, sizeof(int64_t) * (size_t)(R * NSTREAM));
    for (int64_t v = 0; v < n; v++)
        if (g->op_kind[v] == COMM) d->cl[fill[(int64_t)g->op_rank[v] * NSTREAM + g->op_stream[v]]++] = v;
    free(fill);
    free(stream_prev); free(last); free(buf);
    return OK;
nomem:
    free(stream_prev); free(last); free(buf); free_derived(d);
    set_err(err, errlen, "out of memory", 0, 0);
    return E_NOMEM;
}

/* ------------------------------------------------------------------ */
/* One scenario end to end                                              */
/* ------------------------------------------------------------------ */
typedef struct {
    const graph_t *g;
    const derived_t *dv;
    int32_t n_scen, n_refine, n_threads, tid;
    int32_t until_stable, prorate;
    const int64_t *alpha, *bw_intra, *bw_inter, *reduce;
    const uint64_t *jseed;
    const uint32_t *jstream;
    const int32_t *jamp;
    const uint8_t *algo;
    const uint8_t *cc_model;
    const int32_t *cc_table;
    int32_t n_tables;
    const cc_table_t *tables;
    const uint32_t *slow;
    const forest_t *forest;
    int64_t *start, *finish, *step, *cost;
    uint64_t *digest;
    uint32_t *factor;
    int32_t *refinements;
    int rc;
    char msg[256];
} job_t;

static int run_scenario(job_t *jb, int32_t si, work_t *w, int64_t *s, int64_t *f, int64_t *base,
                        int64_t *cost, uint32_t *F, int64_t *O, int64_t *lo_buf, int64_t *hi_buf) {
    const graph_t *g = jb->g;
    const derived_t *dv = jb->dv;
    const int32_t tsel = jb->cc_table ? jb->cc_table[si] : 0;
    if (tsel < 0 || tsel > jb->n_tables) {
        snprintf(jb->msg, sizeof jb->msg, "scenario %d names CC table %d of %d", si, tsel, jb->n_tables);
        return E_RANGE;
    }
    scen_t sc = {jb->alpha[si], jb->bw_intra[si], jb->bw_inter[si], jb->reduce[si], jb->jseed[si],
                 jb->jstream[si], jb->jamp[si], jb->algo[si], jb->cc_model ? jb->cc_model[si] : 0,
                 tsel > 0 ? jb->tables + (tsel - 1) : NULL, jb->slow + (int64_t)si * NCLASS * 4, jb->forest};
    int rc = check_scen(&sc, jb->msg, sizeof jb->msg);
    if (rc) return rc;
    /* CC estimator */
    for (int64_t c = 0; c < g->n_colls; c++) {
        cost[c] = cc_time(g->coll_type[c], g->coll_bytes[c], dv->tN[c], dv->tM[c], dv->tK[c], &sc);
        if (cost[c] < 0) {
            snprintf(jb->msg, sizeof jb->msg, "collective %lld costs >= 2^62 ns", (long long)c);
            return E_RANGE;
        }
    }
    /* pass 1: composer with the (jittered) base durations */
    for (int64_t v = 0; v < g->n_ops; v++) {
        base[v] = g->op_kind[v] == COMM ? 0 : base_duration(g, &sc, v);
        w->dur[v] = base[v];
        F[v] = Q16_ONE;
    }
    rc = compose(g, dv, w->dur, cost, s, f, w, jb->msg, sizeof jb->msg);
    if (rc) return rc;
    /* validator: R refinements, each from the previous pass's timeline; until_stable:
       stop as soon as a refinement would leave every duration unchanged */
    int32_t done = 0;
    for (int32_t p = 0; p < jb->n_refine; p++) {
        overlap_factors(g, dv, &sc, s, f, F, O, lo_buf, hi_buf);
        int changed = 0;
        for (int64_t v = 0; v < g->n_ops; v++) {
            if (g->op_kind[v] != COMPUTE) continue;
            const int64_t d = inflated(base[v], F[v], O[v], jb->prorate);
            changed |= d != w->dur[v];
            w->dur[v] = d;
        }
        if (jb->until_stable && !changed) break;
        rc = compose(g, dv, w->dur, cost, s, f, w, jb->msg, sizeof jb->msg);
        if (rc) return rc;
        done++;
    }
    if (jb->refinements) jb->refinements[si] = done;
    /* step time and digest of the final timeline */
    int64_t step = 0;
    uint64_t dig = 0;
    for (int64_t v = 0; v < g->n_ops; v++) {
        if (f[v] > step) step = f[v];
        dig += mix64(mix64((uint64_t)v ^ (uint64_t)s[v]) ^ (uint64_t)f[v]);
    }
    if (jb->step) jb->step[si] = step;
    if (jb->digest) jb->digest[si] = dig;
    return OK;
}

static void *worker(void *arg) {
    job_t *jb = (job_t *)arg;
    const graph_t *g = jb->g;
    const int64_t n = g->n_ops, nc = g->n_colls;
    work_t w;
    memset(&w, 0, sizeof w);
    w.pending = malloc(sizeof(int64_t) * (size_t)(n + 1));
    w.ready = malloc(sizeof(int64_t) * (size_t)(n + 1));
    w.dur = malloc(sizeof(int64_t) * (size_t)(n + 1));
    w.arrived = malloc(sizeof(int64_t) * (size_t)(nc + 1));
    w.barrier = malloc(sizeof(int64_t) * (size_t)(nc + 1));
    w.heap.a = malloc(sizeof(event_t) * (size_t)(n + 1));
    int64_t *base = malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *s_tmp = jb->start ? NULL : malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *f_tmp = jb->finish ? NULL : malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *c_tmp = jb->cost ? NULL : malloc(sizeof(int64_t) * (size_t)(nc + 1));
    uint32_t *F_tmp = jb->factor ? NULL : malloc(sizeof(uint32_t) * (size_t)(n + 1));
    int64_t *O = malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *lo_buf = malloc(sizeof(int64_t) * (size_t)(n + 1));
    int64_t *hi_buf = malloc(sizeof(int64_t) * (size_t)(n + 1));
    jb->rc = OK;
    if (!w.pending || !w.ready || !w.dur || !w.arrived || !w.barrier || !w.heap.a || !base
        || (!jb->start && !s_tmp) || (!jb->finish && !f_tmp) || (!jb->cost && !c_tmp)
        || (!jb->factor && !F_tmp) || !O || !lo_buf || !hi_buf) {
        jb->rc = E_NOMEM;
        snprintf(jb->msg, sizeof jb->msg, "out of memory");
    }
    for (int32_t si = jb->tid; jb->rc == OK && si < jb->n_scen; si += jb->n_threads) {
        int64_t *s = jb->start ? jb->start + (int64_t)si * n : s_tmp;
        int64_t *f = jb->finish ? jb->finish + (int64_t)si * n : f_tmp;
        int64_t *cost = jb->cost ? jb->cost + (int64_t)si * nc : c_tmp;
        uint32_t *F = jb->factor ? jb->factor + (int64_t)si * n : F_tmp;
        jb->rc = run_scenario(jb, si, &w, s, f, base, cost, F, O, lo_buf, hi_buf);
    }
    free(w.pending); free(w.ready); free(w.dur); free(w.arrived); free(w.barrier); free(w.heap.a);
    free(base); free(s_tmp); free(f_tmp); free(c_tmp); free(F_tmp); free(O); free(lo_buf); free(hi_buf);
    return NULL;
}

/*
 * Entry point.  Scenario fields are structure-of-arrays of length n_scen
 * (slowdown: n_scen x 8 x 4).  Outputs are scenario-major and any may be NULL:
 * start/finish/factor [n_scen][n_ops], cost [n_scen][n_colls], step/digest [n_scen].
 * factor receives the factor found on the timeline before the final pass.
 * Validator options (Sec. 6): until_stable stops refining once a refinement
 * would leave every duration unchanged (at most n_refine refinements;
 * refinements[n_scen] receives how many ran); prorate inflates only the
 * overlapped part of a compute op.
 * Returns 0 or a negative error code; err receives a message.
 */
int oracle_run(int64_t n_ops, int32_t n_ranks, int32_t gpus_per_node, const int32_t *op_rank,
               const uint8_t *op_stream, const uint8_t *op_kind, const uint8_t *op_class,
               const int64_t *op_dur, const int64_t *op_coll, const int64_t *pred_off,
               const int32_t *pred_idx, int64_t n_colls, const uint8_t *coll_type,
               const int64_t *coll_bytes, const int32_t *coll_N, const int32_t *coll_M,
               const int32_t *coll_K, int32_t n_scen, const int64_t *alpha,
               const int64_t *bw_intra, const int64_t *bw_inter, const int64_t *reduce,
               const uint64_t *jseed, const uint32_t *jstream, const int32_t *jamp,
               const uint8_t *algo, const uint8_t *cc_model, const int32_t *cc_table, int32_t n_tables,
               const int64_t *tables, const uint32_t *slow, const void *forest_nodes, int64_t n_nodes,
               const int32_t *forest_roots, int32_t n_trees, int32_t forest_base, const int64_t *class_metrics,
               int32_t n_refine, int32_t until_stable,
               int32_t prorate, int32_t n_threads, int64_t *start, int64_t *finish, int64_t *step,
               uint64_t *digest, int64_t *cost, uint32_t *factor, int32_t *refinements, char *err,
               int64_t errlen) {
    graph_t g = {n_ops, n_ranks, gpus_per_node, op_rank, op_stream, op_kind, op_class, op_dur,
                 op_coll, pred_off, pred_idx, n_colls, coll_type, coll_bytes, coll_N, coll_M, coll_K};
    if ((coll_N || coll_M || coll_K) && !(coll_N && coll_M && coll_K)) {
        set_err(err, errlen, "coll_N, coll_M and coll_K go together", 0, 0);
        return E_ARG;
    }
    if (err && errlen > 0) err[0] = 0;
    if (n_scen < 0 || n_refine < 0 || n_threads < 1) {
        set_err(err, errlen, "bad n_scen %lld / n_refine %lld", (long long)n_scen, (long long)n_refine);
        return E_ARG;
    }
    int rc = check_graph(&g, err, errlen);
    if (rc) return rc;
    const cc_table_t *tb = (const cc_table_t *)tables;
    if (n_tables < 0 || (n_tables > 0 && !tables)) {
        set_err(err, errlen, "bad CC table array", 0, 0);
        return E_ARG;
    }
    for (int32_t k = 0; k < n_tables; k++)
        for (int i = 0; i < CC_ROWS; i++) {
            if (i > 0 && tb[k].max_bytes[i] < tb[k].max_bytes[i - 1]) {
                set_err(err, errlen, "CC table %lld: max_bytes decreases at row %lld", k, i);
                return E_ARG;
            }
            if (tb[k].chunk[i] < 1 || tb[k].chunk[i] >= ((int64_t)1 << 32) || tb[k].alpha[i] < 0
                || tb[k].alpha[i] >= KNOB_LIMIT || tb[k].beta[i] < 0 || tb[k].beta[i] >= KNOB_LIMIT
                || tb[k].gamma[i] < 0 || tb[k].gamma[i] >= KNOB_LIMIT || tb[k].reduce[i] < 1
                || tb[k].reduce[i] >= KNOB_LIMIT) {
                set_err(err, errlen, "CC table %lld row %lld out of range", k, i);
                return E_RANGE;
            }
        }
    /* the ensemble, if any: every tree at most TREE_DEPTH splits deep, indices in range */
    forest_t fo = {(const tree_node_t *)forest_nodes, n_nodes, forest_roots, n_trees, forest_base, class_metrics};
    if (n_trees > 0) {
        if (!forest_nodes || !forest_roots || !class_metrics || n_nodes < 1 || forest_base < (int32_t)Q16_ONE
            || forest_base >= (1 << 20)) {
            set_err(err, errlen, "bad forest (%lld trees, %lld nodes)", n_trees, n_nodes);
            return E_ARG;
        }
        int64_t stack_node[TREE_DEPTH + 2], stack_depth[TREE_DEPTH + 2];
        for (int32_t t = 0; t < n_trees; t++) {
            if (forest_roots[t] < 0 || forest_roots[t] >= n_nodes) {
                set_err(err, errlen, "tree %lld: root %lld out of range", t, forest_roots[t]);
                return E_ARG;
            }
            int sp = 0;
            stack_node[sp] = forest_roots[t];
            stack_depth[sp++] = 0;
            while (sp > 0) {
                const int64_t i = stack_node[--sp], dep = stack_depth[sp];
                const tree_node_t *nd = fo.nodes + i;
                if (nd->feature < 0) continue;
                if (dep >= TREE_DEPTH || nd->feature >= NFEAT || nd->left < 0 || nd->left >= n_nodes
                    || nd->right < 0 || nd->right >= n_nodes) {
                    set_err(err, errlen, "tree %lld: node %lld is malformed or too deep", t, i);
                    return E_ARG;
                }
                stack_node[sp] = nd->left;
                stack_depth[sp++] = dep + 1;
                stack_node[sp] = nd->right;
                stack_depth[sp++] = dep + 1;
            }
        }
    }
    derived_t dv;
    rc = derive(&g, &dv, err, errlen);
    if (rc) return rc;
    if (n_threads > n_scen) n_threads = n_scen > 0 ? n_scen : 1;
    job_t *jobs = calloc((size_t)n_threads, sizeof(job_t));
    pthread_t *th = calloc((size_t)n_threads, sizeof(pthread_t));
    if (!jobs || !th) {
        free(jobs); free(th); free_derived(&dv);
        set_err(err, errlen, "out of memory", 0, 0);
        return E_NOMEM;
    }
    for (int32_t t = 0; t < n_threads; t++) {
        jobs[t] = (job_t){&g, &dv, n_scen, n_refine, n_threads, t, until_stable != 0, prorate != 0, alpha,
                          bw_intra, bw_inter, reduce, jseed, jstream, jamp, algo, cc_model, cc_table, n_tables, tb,
                          slow, n_trees > 0 ? &fo : NULL, start, finish, step, cost, digest, factor, refinements,
                          OK, {0}};
    }
    for (int32_t t = 1; t < n_threads; t++) pthread_create(&th[t], NULL, worker, &jobs[t]);
    worker(&jobs[0]);
    for (int32_t t = 1; t < n_threads; t++) pthread_join(th[t], NULL);
    rc = OK;
    for (int32_t t = 0; t < n_threads; t++)
        if (jobs[t].rc != OK) {
            rc = jobs[t].rc;
            if (err && errlen > 0) snprintf(err, (size_t)errlen, "%s", jobs[t].msg);
            break;
        }
    free(jobs); free(th); free_derived(&dv);
    return rc;
}

/* Exposed pieces for the pin tests (each is the oracle's own code above). */
int64_t oracle_chunk_bytes(int64_t S) { return chunk_bytes(S); }
int64_t oracle_cc_time(int32_t type, int64_t S, int64_t N, int64_t M, int64_t K, int64_t alpha,
                       int64_t bw_intra, int64_t bw_inter, int64_t reduce, int32_t algo, int32_t cc_model,
                       const int64_t *table) {
    uint32_t slow[32];
    for (int i = 0; i < 32; i++) slow[i] = Q16_ONE;
    scen_t sc = {alpha, bw_intra, bw_inter, reduce, 0, 0, 0, (uint8_t)algo, (uint8_t)cc_model,
                 (const cc_table_t *)table, slow, NULL};
    return cc_time(type, S, N, M, K, &sc);
}
uint64_t oracle_splitmix64_at(uint64_t seed, uint64_t k) { return splitmix64_at(seed, k); }
int64_t oracle_q16(int64_t d, uint64_t f) { return q16_scale(d, f); }
uint64_t oracle_mix64(uint64_t z) { return mix64(z); }
