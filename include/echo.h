/*
 * echo.h -- C ABI of the MI355X timeline composer (libecho.so).
 *
 * The library implements the simulation hot path of Echo (arXiv 2412.12487):
 * given the per-rank execution graphs of a distributed training job, it costs
 * every collective with the white-box CC model (Sec. 5.3, Eq. 1-5, Table 6),
 * composes global per-op timelines across all ranks (Sec. 4.2) with the
 * collective synchronisation rule of Sec. 5.2, inflates computation kernels
 * that overlap communication by a slowdown factor (Sec. 6 and the slowdown
 * definition next to Table 2) and recomposes.  Many what-if scenarios are
 * evaluated in one call, one GPU lane per scenario.
 *
 * Conventions for every entry point:
 *   - return 0 (ECHO_OK) or a negative ECHO_ERR_* code; nothing throws;
 *   - echo_last_error() returns a message for the calling thread's last error;
 *   - "host" pointers are read during the call only and may be freed after it;
 *   - "device" pointers are HIP device memory owned by the caller and must
 *     stay valid until the enqueued work has finished;
 *   - all device work is enqueued asynchronously on the caller's HIP stream
 *     (hipStream_t passed as void*, NULL = the null stream);
 *   - times are int64 nanoseconds; slowdown factors are Q16 fixed point
 *     (65536 = 1.0).
 */
#ifndef ECHO_H
#define ECHO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes. */
enum {
    ECHO_OK = 0,
    ECHO_ERR_ARG = -1,    /* malformed argument or graph structure               */
    ECHO_ERR_RANGE = -2,  /* a value outside the documented ranges, or a time >= 2^62 */
    ECHO_ERR_MATCH = -3,  /* collective membership breaks the matching rules      */
    ECHO_ERR_CYCLE = -4,  /* the merged graph has a cycle: the simulated job deadlocks */
    ECHO_ERR_NOMEM = -5,  /* host or device allocation failed                     */
    ECHO_ERR_HIP = -6,    /* a HIP runtime call failed                            */
    ECHO_ERR_DEVICE = -7  /* a device-side check failed (see echo_sync_status)    */
};

/* Operator kinds, collective types and all-reduce algorithms. */
enum { ECHO_COMPUTE = 0, ECHO_COMM = 1, ECHO_MEMCPY = 2 };
enum { ECHO_AR = 0, ECHO_AG = 1, ECHO_RS = 2, ECHO_P2P = 3 };
enum { ECHO_RING = 0, ECHO_TREE = 1 };

typedef struct echo_graph_s *echo_graph;

/*
 * Per-rank execution graphs of one training step, as the paper's workload
 * tracer produces them (Sec. 4.1): operators with dependencies and measured
 * durations, communication operators as placeholders naming their group
 * and message size.  All arrays are host memory owned by the caller.
 *
 *   n_ops          number of operators, 0 <= n_ops < 2^31
 *   op_rank[n]     rank issuing the op, 0 <= rank < n_ranks; non-decreasing:
 *                  ops are rank-major and, within a rank, in program order
 *   op_stream[n]   stream on that rank, 0..7.  Ops of one stream run FIFO in
 *                  program order (each waits for the previous one to finish)
 *   op_kind[n]     ECHO_COMPUTE, ECHO_COMM or ECHO_MEMCPY
 *   op_class[n]    kernel class 0..7: the row of the slowdown table
 *   op_dur_ns[n]   base duration of compute/memcpy ops, 0 <= d < 2^43; ignored for comm
 *   op_coll[n]     collective id of a comm op (0 <= id < n_colls), -1 otherwise
 *   pred_off[n+1], pred_idx[pred_off[n]]
 *                  explicit dependencies of op v: pred_idx[pred_off[v] ..
 *                  pred_off[v+1]-1], each an earlier op of the same rank.
 *                  Cross-rank coupling exists only through collectives.
 *   n_colls        number of collectives
 *   coll_type[c]   ECHO_AR, ECHO_AG, ECHO_RS or ECHO_P2P
 *   coll_bytes[c]  message size S, 0 <= S < 2^50 (AG/RS: the full buffer)
 *   gpus_per_node  ranks per server: node(rank) = rank / gpus_per_node
 *   coll_N[c], coll_M[c], coll_K[c]
 *                  optional (all three or none; NULL = derived from the members):
 *                  the membership the cost of collective c is computed with --
 *                  N members, M distinct servers, K most members on one server --
 *                  when some members are not part of this graph.  This is the
 *                  symmetry reduction of data-parallel training (Sec. 8.5, DDP
 *                  mode: one copy of the workload per DP group): simulate one DP
 *                  replica, give each collective its whole group's N, M, K, and
 *                  its barrier is met by the member ops present (a DP collective
 *                  with one local member becomes a self-barrier).  When every
 *                  replica has the same durations (no jitter) the result equals
 *                  the sweep over all replicas op for op.  Requires
 *                  1 <= M <= N, 1 <= K <= N, M*K >= N, N >= the members present,
 *                  N = 2 for P2P; else ECHO_ERR_ARG.
 *
 * Collective membership is explicit (op_coll): every rank in a group joins
 * with exactly one comm op.  P2P collectives have exactly two members.
 */
typedef struct {
    int64_t n_ops;
    int32_t n_ranks, gpus_per_node;
    const int32_t *op_rank;
    const uint8_t *op_stream, *op_kind, *op_class;
    const int64_t *op_dur_ns;
    const int64_t *op_coll;
    const int64_t *pred_off;
    const int32_t *pred_idx;
    int64_t n_colls;
    const uint8_t *coll_type;
    const int64_t *coll_bytes;
    const int32_t *coll_N, *coll_M, *coll_K;
} echo_graph_desc;

/*
 * One what-if scenario (192 bytes; callers pass a device array of these).
 *   alpha_ns          connection set-up time alpha, 0 <= alpha < 2^40
 *   bw_intra_MBps     intra-server bandwidth; beta = ceil(chunk*1000 / bw_intra)
 *   bw_inter_MBps     inter-server bandwidth; gamma = ceil(chunk*1000 / bw_inter)
 *   reduce_MBps       reduction throughput; reduce time = ceil(S*1000 / reduce)
 *                     (each of the three in [1, 2^40))
 *   jitter_seed, jitter_stream, jitter_amp_q16
 *                     optional per-op duration jitter of amplitude A (Q16,
 *                     0 <= A <= 65535, 0 = off): D(v) = q16(d(v), 65536 + J) with
 *                     J = floor((u >> 32) * (2A+1) / 2^32) - A, u the k-th output of
 *                     SplitMix64 seeded with jitter_seed, k = jitter_stream*2^36 + v + 1
 *   ar_algo           ECHO_RING or ECHO_TREE for all-reduce collectives
 *   cc_model          ECHO_CC_ECHO (0): the chunked model of Eq. 2-5;
 *                     ECHO_CC_ALPHA_BETA (1): the alpha-beta baseline (see below)
 *   cc_table          0: Eq. 2-5 take chunk sizes from Table 6 and beta, gamma and
 *                     the reduce time from the three bandwidths above; k >= 1:
 *                     they come from row set k-1 of the graph's CC parameter tables
 *                     (echo_set_cc_tables), alpha included
 *   slowdown_q16[k][t] factor for a class-k compute op overlapping a type-t
 *                     collective, 65536 <= f < 2^20
 * q16(d, f) = (d*f + 32768) >> 16 in unsigned 64-bit arithmetic.
 *
 * Alpha-beta baseline (a what-if reference, not the paper's model): the
 * latency-bandwidth cost of the ring and binomial-tree algorithms (Thakur,
 * Rabenseifner and Gropp, IJHPCA 2005) with one rounding per step.  With
 * B = bw_inter if the group spans servers else bw_intra, R = reduce,
 * t_B(x) = ceil(x*1000 / B), t_R(x) = ceil(x*1000 / R), p = ceil(S / N),
 * L = ceil(log2 N):  AG (N-1)(alpha + t_B(p));  RS (N-1)(alpha + t_B(p) + t_R(p));
 * ring AR (N-1)(2 alpha + 2 t_B(p) + t_R(p));  tree AR L(2 alpha + 2 t_B(S) + t_R(S));
 * P2P alpha + t_B(S).
 */
typedef struct {
    int64_t alpha_ns, bw_intra_MBps, bw_inter_MBps, reduce_MBps;
    uint64_t jitter_seed;
    uint32_t jitter_stream;
    int32_t jitter_amp_q16;
    uint8_t ar_algo;
    uint8_t cc_model;
    uint8_t pad0[2];
    int32_t cc_table;
    uint8_t pad1[8];
    uint32_t slowdown_q16[8][4];
} echo_scenario;

enum { ECHO_CC_ECHO = 0, ECHO_CC_ALPHA_BETA = 1 };

/*
 * CC parameter table (Sec. 5.3 offline profiling: per chunk size, the
 * connection set-up time, intra- and inter-server transmission times and the
 * reduce throughput; Table 6 lists such rows by tensor size).  Row i serves
 * collectives with S <= max_bytes[i] (the first such row; the last row also
 * every larger S).  Per row: chunk size in bytes (1 <= chunk < 2^32), alpha,
 * beta and gamma in ns (per chunk for beta and gamma, each in [0, 2^40)) and
 * the reduce throughput in MB/s ([1, 2^40)).  max_bytes must not decrease.
 */
#define ECHO_CC_ROWS 7
typedef struct {
    int64_t max_bytes[ECHO_CC_ROWS];
    int64_t chunk[ECHO_CC_ROWS];
    int64_t alpha_ns[ECHO_CC_ROWS];
    int64_t beta_ns[ECHO_CC_ROWS];
    int64_t gamma_ns[ECHO_CC_ROWS];
    int64_t reduce_MBps[ECHO_CC_ROWS];
} echo_cc_table;

/*
 * Validate a graph, match its collectives, merge each collective into one
 * barrier node, order the merged graph by topological level and upload it
 * to device `hip_device` (the analogue of the simulator's initialisation,
 * Sec. 8.5, Table 8).  Matching rule (Sec. 4.2: predefined matching rules
 * plus a user API): within one communicator -- the set of (rank, stream) of a
 * collective's members -- every member rank issues that communicator's
 * collectives in the same order.  Errors: ARG (malformed arrays), RANGE,
 * MATCH (a rank with two members of one collective, a P2P collective without
 * exactly two members, a collective with no member, or an issue-order
 * mismatch), CYCLE (deadlocked job), NOMEM, HIP.  The caller's arrays are
 * copied; on success *out owns host and device memory until echo_free_graph.
 */
int echo_load_graph(const echo_graph_desc *desc, int hip_device, echo_graph *out);

/*
 * echo_load_graph with an explicit walker width.  The composer walks each
 * scenario tile with one wavefront per "walker" -- `ranks_per_walker`
 * consecutive ranks whose ops it visits in level order -- and every walker of
 * a tile must be resident on the device at once.  0 picks the fewest ranks
 * per walker that fit (one, unless the graph has more ranks than the device
 * holds wavefronts); a positive value asks for at least that many (up to 16).
 * Results do not depend on it.  Errors: as echo_load_graph; ARG for a value
 * outside [0, 16]; RANGE when the graph does not fit at 16 ranks per walker.
 */
int echo_load_graph_ex(const echo_graph_desc *desc, int hip_device, int32_t ranks_per_walker, echo_graph *out);

/* Sizes of a loaded graph: ops, collectives and topological levels of the merged graph. */
int echo_graph_info(echo_graph g, int64_t *n_ops, int64_t *n_colls, int64_t *n_levels);

/* Release a graph (waits for the device to be idle first).  NULL is allowed. */
void echo_free_graph(echo_graph g);

/*
 * Give the graph n_tables CC parameter tables (host array, copied; n_tables = 0
 * removes them).  Scenarios select one with cc_table = index + 1; a scenario
 * naming a table the graph does not have is reported by echo_sync_status
 * (ECHO_ERR_RANGE).  Errors: ARG (NULL with n_tables > 0, n_tables < 0,
 * decreasing max_bytes), RANGE (a value outside its range), NOMEM, HIP.
 */
int echo_set_cc_tables(echo_graph g, const echo_cc_table *tables, int32_t n_tables);

/*
 * CC estimator (Sec. 5.3): d_cost[c * n_scen + s] = running time of collective
 * c under scenario s -- ring AG (Eq. 2), ring RS (Eq. 3), ring or tree AR
 * (Eq. 4, Eq. 5) and P2P as one chunked hop -- with chunk sizes of Table 6.
 * N = members, M = distinct servers among them, K = most members on one
 * server.  d_scen: device, n_scen records.  d_cost: device, n_colls * n_scen
 * int64.  Scenario ranges are checked on the device (echo_sync_status).
 */
int echo_cc_cost(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int64_t *d_cost,
                 void *hip_stream);

/*
 * Compose the timelines of every scenario.  Pass 1 composes with the base
 * (jittered) durations: op v waits for all its predecessors (stream FIFO and
 * explicit dependencies); a comm op starts at its own launch and finishes when
 * the last member of its collective has launched plus the collective's cost
 * (Sec. 5.2).  Each of the n_refine >= 0 refinements then inflates every
 * compute op that overlapped a comm op of the same rank in the previous pass
 * -- duration q16(D, F) with F the largest slowdown_q16[class][type] over the
 * overlapping comm ops -- and composes again from the base durations.
 * Outputs (device, caller-owned, any of start/finish/digest may be NULL):
 *   d_start[v * n_scen + s], d_finish[v * n_scen + s]  final-pass timeline
 *   d_step[s]    step time: the latest finish of any op
 *   d_digest[s]  sum over ops (mod 2^64) of mix(mix(v ^ start) ^ finish),
 *                mix = the SplitMix64 output function
 * Works on the device only; range violations found there are reported by
 * echo_sync_status.  Calls on one graph must not overlap (they share its
 * workspace); the workspace grows on demand (hipMalloc) and is freed with
 * the graph.  The call enqueues kernels only (no memset, no host
 * synchronisation), so once an eager call with at least as many scenarios
 * and the same options has sized the workspace, it can be recorded by HIP
 * stream capture and replayed as a graph (kernel timing must be off).
 * The walk runs as cooperative launches (every wavefront of a launch
 * resident at once).  Observed on MI355X: once one process has made such
 * launches on a GPU, another process's are refused and the call returns
 * ECHO_ERR_HIP, so compose from one process per GPU.
 */
int echo_compose_batch(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int32_t n_refine,
                       int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                       void *hip_stream);

/*
 * Validator options (Sec. 3 and Sec. 6 give the model -- overlapped
 * computation runs slower -- but no iteration rule).
 *   max_refine    at most this many refinements (0..64)
 *   until_stable  nonzero: stop refining a scenario once a refinement would
 *                 leave every duration unchanged (the timeline is then a fixed
 *                 point: one more refinement reproduces it)
 *   prorate       nonzero: inflate only the overlapped part of a compute op:
 *                 duration D - o + q16(o, F), o = the time of [start, finish)
 *                 covered by the union of the overlapping comm ops' intervals
 *                 on the previous timeline, capped at D; zero: q16(D, F)
 *   forest        nonzero: F comes from the graph's tree ensemble
 *                 (echo_set_forest) instead of the scenario's slowdown table
 */
typedef struct {
    int32_t max_refine;
    int32_t until_stable;
    int32_t prorate;
    int32_t forest;
} echo_validator;

/*
 * Slowdown prediction by a gradient-boosted tree ensemble (Sec. 6: an
 * XGBoost regressor over communication details and computation-kernel
 * metrics, Table 4; trees at most 12 splits deep, Table 5).  For a compute op
 * v overlapped by comm ops of collective type t, the feature vector is
 *   x[0] kernel class   x[1] base duration d0 (ns; the profiled running time)
 *   x[2] t              x[3] largest message S among the overlapping type-t ops
 *   x[4] most members N among them (the N their cost uses)
 *   x[5] the scenario's ar_algo   x[6] bw_intra_MBps   x[7] bw_inter_MBps
 *   x[8..11] class_metrics[class][0..3] (kernel metrics of the class)
 * and the prediction is base_q16 plus one leaf value per tree -- each tree
 * walked from its root, left when x[feature] < threshold -- kept inside
 * [65536, 2^20).  F(v) is the largest prediction over the collective types
 * overlapping v.  Integer features, thresholds and leaves: bit-exact.
 */
typedef struct {
    int32_t feature;    /* 0..11, or -1 for a leaf */
    int32_t left, right;/* children: node indices */
    int32_t value;      /* leaf: contribution to the factor (Q16) */
    int64_t threshold;
} echo_tree_node;
#define ECHO_TREE_DEPTH 12

/*
 * Give the graph a tree ensemble (host arrays, copied): n_nodes nodes, the
 * roots of n_trees trees, the base score (65536 <= base < 2^20) and
 * class_metrics[8][4].  Every root-to-leaf path has at most ECHO_TREE_DEPTH
 * splits.  n_trees = 0 removes the ensemble.  Errors: ARG (malformed trees or
 * arrays), RANGE (more than 2^26 nodes once every tree is laid out on its own,
 * nodes shared between paths copied), NOMEM, HIP; on ARG and RANGE the graph
 * keeps its previous ensemble.
 */
int echo_set_forest(echo_graph g, const echo_tree_node *nodes, int64_t n_nodes, const int32_t *roots,
                    int32_t n_trees, int32_t base_q16, const int64_t *class_metrics);

/*
 * echo_compose_batch with validator options.  d_refinements (device, n_scen
 * int32, or NULL) receives the refinements composed per scenario: with
 * until_stable, those that changed some duration; else max_refine.  Passes
 * past the point where every scenario is stable are skipped on the device
 * (no host synchronisation).  With prorate, the extra time of one op,
 * q16(o, F) - o, must stay below 2^32 - 1 ns (else ECHO_ERR_RANGE from
 * echo_sync_status).  Errors and ownership as echo_compose_batch; ARG for a
 * NULL options pointer, max_refine outside 0..64 or forest without an ensemble.
 */
int echo_compose_validated(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, const echo_validator *opts,
                           int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                           int32_t *d_refinements, void *hip_stream);

/*
 * Wait for `hip_stream` and report the device-side status of the graph's
 * launches since the previous call: ECHO_OK, ECHO_ERR_RANGE (a scenario knob
 * out of range or a time >= 2^62) or ECHO_ERR_DEVICE (a wait for a collective
 * exceeded the spin limit).  Clears the status.
 */
int echo_sync_status(echo_graph g, void *hip_stream);

/*
 * Optional per-kernel timing of echo_compose_batch: when enabled, HIP events
 * are recorded on the caller's stream around every kernel the call launches.
 * echo_kernel_times (after the stream has finished, e.g. after
 * echo_sync_status) reports the last compose call's kernels in launch order:
 * kinds[i] is ECHO_K_* and ms[i] the event-measured duration.  *n receives the
 * number of kernels (at most max are written).
 */
enum { ECHO_K_INIT = 0, ECHO_K_CC_COST = 1, ECHO_K_WALK = 2, ECHO_K_OVERLAP = 3, ECHO_K_CLEAR = 4 };
int echo_set_timing(echo_graph g, int enable);
int echo_kernel_times(echo_graph g, int32_t max, int32_t *kinds, float *ms, int32_t *n);

/*
 * Bounded waits.  A composer wavefront that waits for the members of a
 * collective gives up after limit_ns nanoseconds of wall clock (default 20 s;
 * counted from the wait's 16th poll of device memory or 256th poll of LDS):
 * it sets the graph's timeout status, every other wait of the launch gives
 * up too, and every kernel runs to its end (the timelines it writes are then
 * meaningless) -- echo_sync_status reports ECHO_ERR_DEVICE.  The limit applies
 * to each wait, not to a whole call; it is read when a compose is enqueued.
 * 10 <= limit_ns <= 2^40 (the device clock ticks every 10 ns).  Errors: ARG.
 */
int echo_set_spin_limit(echo_graph g, int64_t limit_ns);

/*
 * Scenario tiles per walk launch.  The composer walks all scenario tiles of a
 * pass in as few cooperative launches as the device holds co-resident (every
 * walker of a tile must run at once); max_tiles > 0 caps the tiles of one
 * launch (a pass then takes more launches), 0 restores the default.  Results
 * do not depend on it.  Errors: ARG for max_tiles < 0.
 */
int echo_set_launch_tiles(echo_graph g, int32_t max_tiles);

/*
 * Latency floor of the composer's walk (analysis; reads host-side copies of
 * the walk lists, no device work).  Each scenario tile is walked by one
 * wavefront per walker, which visits its walk list in order; a comm op's
 * finish is taken at its resolve item, which waits until every member's
 * launch item has run.  With weight_ps[0] picoseconds per item, plus
 * weight_ps[1] for a resolve item whose barrier is met in LDS (all members in
 * one workgroup) or weight_ps[2] for one met in device memory, out receives
 * the longest chain through those dependencies:
 *   out[0] its length in picoseconds, out[1] its items, out[2] its
 *   LDS-barrier and out[3] its device-memory-barrier resolve items.
 * Weights in [0, 2^40).  Errors: ARG.
 */
int echo_walk_chain(echo_graph g, const int64_t weight_ps[3], int64_t out[4]);

/*
 * echo_compose_batch for callers that cannot allocate device memory: code
 * under HIP stream capture, serving loops or harnesses that forbid hipMalloc.
 * It composes exactly as echo_compose_batch (the same kernels, bit-identical
 * results) but takes its workspace -- the per-scenario cost-class table,
 * barrier arrival maxima, counts and member slots, and the overlap masks of the refined
 * passes -- from one fixed device array of ECHO_SCRATCH_BYTES per GPU, which
 * the library holds from the first echo_load_graph on that GPU until the
 * process ends, and it allocates nothing.  The caller passes every output:
 * d_start and d_finish ([n_ops][n_scen] int64) and d_step are required (the
 * walk keeps its working times there); d_digest may be NULL.  Kernel timing
 * (echo_set_timing) is not recorded.  The workspace, each part rounded up to
 * 256 bytes, is 8 * n_classes * n_scen (cost classes) + 8 * n_counted * n_scen
 * (arrivals) + 4 * n_counted * ceil(n_scen / 64) (counts; n_counted: the
 * collectives of more than eight members met in device memory, not in one
 * workgroup) + 8 * n_slots * n_scen (n_slots: the member ops of collectives of
 * at most eight members met in device memory) + with n_refine > 0
 * (n_items + 32) * 65 * ceil(n_scen / 64) bytes (masks and a flag byte per
 * row and tile; n_items = ops + comm ops); a call needing more returns
 * ECHO_ERR_RANGE before enqueuing anything.
 * Every call on one GPU shares that GPU's array: calls whose work overlaps on
 * the device (two streams, two threads, two graphs) race and must be
 * serialised by the caller.  Errors: as echo_compose_batch, plus ARG for a
 * NULL d_start, d_finish or d_step and HIP if the array is unavailable.
 */
#define ECHO_SCRATCH_BYTES ((int64_t)64 << 20)
int echo_compose_batch_static(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int32_t n_refine,
                              int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                              void *hip_stream);

/* Message of the calling thread's last error ("" if none). */
const char *echo_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ECHO_H */
