// echo_internal.h -- device data layout and kernel launchers of libecho.so.
//
// The loader turns the caller's per-rank graphs into one "walk list" per
// walker: a walker is a group of consecutive ranks (one rank unless the graph
// has more ranks than the device holds co-resident wavefronts), and its list
// holds their ops ordered by (key, rank, program order) where key is the op's
// topological level in the merged graph (a collective merged into one barrier
// node) -- for a comm op, the level at which it can launch.  A wavefront walks
// one walker for 64 scenarios (one lane each); predecessors that are the
// latest op of a register slot stay in registers, the rest are read back from
// the finish array.  Collective barriers are met through per-(collective,
// scenario) arrival maxima and per-(collective, scenario tile) arrival counts,
// or in LDS when every member sits in one workgroup.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "echo.h"

namespace echo {

constexpr int kStreams = 8;
constexpr int kClasses = 8;
constexpr int kTypes = 4;
constexpr int kLanes = 64;                       // scenarios per wavefront
constexpr int64_t kTimeLimit = int64_t(1) << 62;

// Device status bits (per graph).
constexpr unsigned kStatusRange = 1u;            // scenario knob out of range
constexpr unsigned kStatusOverflow = 2u;         // a time reached 2^62
constexpr unsigned kStatusTimeout = 4u;          // a barrier wait exceeded the spin limit
constexpr unsigned kStatusAbort = 8u;            // stop all waits (set with timeout)

// One entry of a walk list (32 bytes, read wave-uniformly).  The (rank,
// stream) pairs of a walker are mapped to eight register "slots": slot 0 is
// its busiest compute/memcpy stream, so most items only touch slot 0.  Pairs
// left without a slot (a walker of several ranks) keep nothing in registers:
// their ops carry kNoReg and their successors read them back from memory.
// A comm op's launch item publishes its arrival; a resolve item placed right
// before its first successor waits for the barrier and writes its finish (to its
// slot, or only to memory without one).
struct WalkItem {
    int32_t op;         // op id: row of the [op][scenario] outputs
    uint32_t meta;      // kind | slot << 2 | class << 5 | regmask << 8 | fast << 16 | noreg << 17
                        // | need start << 18 | need finish << 19 | fold << 20
    int32_t far_off;    // predecessors read back from memory: far[far_off .. +nfar)
    int32_t coll;       // collective of a comm op, -1 otherwise; of a collective met by counting
                        // arrivals in device memory (neither in LDS nor through member slots),
                        // its index among those collectives
    int64_t dur;        // base duration of compute / memcpy ops; resolve item: cost class
    int32_t nfar;
    int32_t aux;
};
static_assert(sizeof(WalkItem) == 32, "walk item must stay 32 bytes");

// A "fast" item is a compute/memcpy op on slot 0 whose start is slot 0's value:
// its only predecessors are the previous op of slot 0 and comm ops whose resolve
// items, right before it, folded their finishes into slot 0 (kFold).
constexpr uint32_t kFast = 1u << 16;
// The op's (rank, stream) pair has no register slot.
constexpr uint32_t kNoReg = 1u << 17;
// A pass that does not produce the caller's timelines stores only what later
// steps read back: the start (kNeedS) of comm ops and of compute ops that do not
// simply follow the previous compute op of their stream (overlap detection
// rebuilds the others), and the finish (kNeedF) of comm ops and of ops read as
// far predecessors.
constexpr uint32_t kNeedS = 1u << 18;
constexpr uint32_t kNeedF = 1u << 19;
// Resolve item: after writing the comm op's finish, raise slot 0 to it.
constexpr uint32_t kFold = 1u << 20;
// Item kind (besides compute/comm/memcpy) that finishes a kNoReg comm op:
// wait for its barrier, then write its finish.
constexpr int kResolve = 3;

// Workgroups walk kBlockWalkers consecutive walkers (one wavefront each) for
// one scenario tile.  A collective whose members all sit in one block is met in
// LDS: each communicator of the block owns a channel with two alternating
// slots (max of launch times per lane, arrival count).  Collective costs are
// looked up per cost class -- the (type, S, N, M, K) tuple that fixes T(c, s)
// for a scenario -- and a block stages its most used classes in LDS.
constexpr int kBlockWalkers = 8;
constexpr int kFlagRowTiles = 2;    // final mask passes of this many tiles per launch fetch only flagged rows
constexpr int kBlock = 32;          // walk items fetched (and overlap masks staged) per round
constexpr int kChannels = 8;          // LDS barrier channels per block
constexpr int kClassSlots = 8;        // LDS cost classes per block
constexpr uint32_t kNoSlot = 15;
// Comm item aux word: bit 0 local barrier | channel << 1 | slot parity << 4 |
// class slot << 5 (kNoSlot: read the class's cost from global memory) | expected count << 9.
constexpr uint32_t kAuxLocal = 1u;
constexpr int kExpectedBits = 23;
// A collective met in device memory whose members are few (at most kSlotMembers)
// meets through per-member slots: each member's launch item stores its launch time
// into its own slot (cleared to -1 before every pass), and a resolve item reads all
// its collective's slots -- a value of -1 means "not yet launched".  The launch item
// carries its slot in `dur`, the resolve item the collective's first slot in
// `far_off`; aux bit 1 marks the mode and the expected-count field holds the member
// count.  Larger collectives count their arrivals and keep a per-scenario maximum.
constexpr uint32_t kAuxSlots = 2u;
constexpr int kSlotMembers = 8;
__host__ __device__ inline int aux_channel(uint32_t x) { return int((x >> 1) & 7u); }
__host__ __device__ inline int aux_parity(uint32_t x) { return int((x >> 4) & 1u); }
__host__ __device__ inline int aux_slot(uint32_t x) { return int((x >> 5) & 15u); }
__host__ __device__ inline unsigned aux_expected(uint32_t x) { return x >> 9; }

__host__ __device__ inline int item_kind(uint32_t m) { return int(m & 3u); }
__host__ __device__ inline int item_stream(uint32_t m) { return int((m >> 2) & 7u); }
__host__ __device__ inline int item_class(uint32_t m) { return int((m >> 5) & 7u); }
__host__ __device__ inline unsigned item_regmask(uint32_t m) { return (m >> 8) & 0xffu; }

// Overlap detection records, per compute op and scenario, which collective
// types overlap it as a 4-bit mask (bit t: some comm op of type t on the same
// rank overlaps).  The slowdown factor is the largest table entry
// slowdown_q16[class][t] over the set bits, 65536 for an empty mask.
// Compute op of a (rank, stream) list for overlap detection (16 bytes).
struct ComputeRec {
    int32_t op;
    uint32_t meta;      // class | kChained
    int64_t dur;        // base duration
};
static_assert(sizeof(ComputeRec) == 16, "compute record must stay 16 bytes");
// Compute op whose only predecessor is the previous compute op of its stream:
// it starts exactly when that op finishes.
constexpr uint32_t kChained = 0x80;
// Overlap detection checks compute ops in blocks of kOverlapBlock (per (rank, stream)
// list, from its start): the walk stores the finish of every block's last op, and a
// block that ends before every comm cursor starts overlaps nothing.
constexpr int kOverlapBlock = 8;

// Inputs of the CC model for a table of collectives (or of cost classes).
struct CollTable {
    int64_t n = 0;
    int64_t *bytes = nullptr;        // S
    int64_t *chunk = nullptr;        // chunk size (Table 6)
    int64_t *eta_ring = nullptr;     // ceil(S / (N * chunk))
    int64_t *eta_chunks = nullptr;   // ceil(S / chunk)
    int32_t *N = nullptr, *M = nullptr, *K = nullptr;
    uint8_t *type = nullptr;
};

// Device copy of a loaded graph (all pointers are device memory).
// Device form of a tree node, one 16-byte load: the two children of a split sit side
// by side, and the walk goes to left + (x >= threshold).  A leaf loops to itself
// (threshold INT64_MIN, left = its own index - 1), so every tree is walked exactly
// ECHO_TREE_DEPTH steps without a branch; leaf values live in a separate array.
struct DevTreeNode {
    int64_t threshold;
    int32_t feature;
    int32_t left;
};
static_assert(sizeof(DevTreeNode) == 16, "one 16-byte load per node");

// Compact form of the ensemble, held in LDS while overlap detection runs.  Features are
// compared by bin: for feature f the ensemble's split thresholds, sorted and without
// repeats, are T_f[0 .. K_f); the bin of a value x is the number of them <= x, so
// "x < T_f[r]" holds exactly when bin(x) <= r.  A node is one 32-bit word laid out like
// DevTreeNode (breadth first per tree, a split's children side by side): feature
// (bits 0-3), the rank r of its threshold in T_f (bits 4-17), left child minus its own
// index (bits 18-31; right = left + 1).  A leaf has feature kFxLeaf and its value in
// bits 4-31 (signed); its feature's bin is always 0, so it loops to itself.
constexpr int kFxFeatures = 12;
constexpr uint32_t kFxLeaf = 15;
constexpr int kFxRows = 16;                  // bin rows per lane; rows 12..15 stay 0
constexpr int kFxMaxWords = 12 * 1024;       // LDS budget of the nodes (48 KB of a 64 KB workgroup, roots aside)
constexpr int kFxRankBits = 14;
struct CompactForest {
    uint32_t *words = nullptr;               // [n_words]
    int32_t n_words = 0;                     // 0: no compact form (the ensemble does not fit)
    int64_t *thr = nullptr;                  // every feature's thresholds, concatenated
    int32_t thr_off[kFxFeatures + 1] = {};   // feature f: thr[thr_off[f] .. thr_off[f + 1])
    int32_t *cbin = nullptr;                 // [class][kFxFeatures]: bins of the class's own features
    int32_t tbin[4] = {};                    // bin of each collective type
    int32_t *coll_bin = nullptr;             // [coll][2]: bins of S and of the N its cost uses
    int32_t *cp_bin = nullptr;               // [compute record]: bin of the base duration
};

struct DeviceGraph {
    int64_t n_ops = 0, n_colls = 0;
    int32_t n_ranks = 0, n_walkers = 0, n_blocks = 0;
    WalkItem *items = nullptr;       // walk lists, walker-major
    int64_t *walk_off = nullptr;     // [n_walkers + 1] offsets into items
    int32_t *far = nullptr;          // far predecessor op ids
    CollTable colls;                 // every collective
    int32_t *members = nullptr;      // [n_colls] member ops present: arrivals that complete a barrier
    CollTable classes;               // every cost class
    int32_t *block_class = nullptr;  // [n_blocks][kClassSlots] class staged in each LDS slot, -1 = none
    // overlap detection: comm / compute ops of each (rank, stream), program order
    int64_t *cl_off = nullptr;       // [n_ranks * 8 + 1]
    int32_t *cl = nullptr;
    uint8_t *cl_type = nullptr;      // collective type of each listed comm op
    int64_t *cp_off = nullptr;       // [n_ranks * 8 + 1]
    ComputeRec *cp = nullptr;
    int32_t *cp_pos = nullptr;       // [compute record] position of the op's item in the walk lists
    unsigned *status = nullptr;      // device status word
    echo_cc_table *cc_tables = nullptr;   // CC parameter tables (echo_set_cc_tables)
    int32_t n_cc_tables = 0;
    int32_t *cl_coll = nullptr;      // collective of each listed comm op (parallel to cl)
    // slowdown ensemble (echo_set_forest)
    DevTreeNode *forest_nodes = nullptr;
    int32_t *forest_leaf = nullptr;  // [node] value of a leaf (0 for a split)
    int32_t *forest_roots = nullptr;
    int64_t *class_metrics = nullptr;  // [8][4]
    int32_t n_trees = 0, forest_base = 65536;
    CompactForest fx;                  // the ensemble in LDS form, when it fits
    int32_t max_comm_streams = 0;    // the most streams with comm ops on one rank
    int64_t n_slots = 0;             // member slots of the collectives met through slots
    int64_t n_counted = 0;           // collectives met by counting arrivals in device memory
    int32_t *counted_members = nullptr;   // [n_counted] their member ops present
};

constexpr int kClassMetrics = 4;

struct WalkArgs {
    const WalkItem *items;
    const int64_t *walk_off;
    const int32_t *far;
    const int32_t *c_N;              // [counted coll] member ops present (arrivals that complete the barrier)
    const int32_t *block_class;
    const echo_scenario *scen;
    const int64_t *class_cost;       // [class][scen]
    // Per-item outputs of overlap detection, one row per walk item (rows of items that are
    // not compute ops unused), mstride columns (the tiles' scenarios, padded to whole tiles):
    const uint8_t *tmask;            // overlap type masks, or null (pass 1)
    const uint32_t *ext;             // extra times (prorating, ensemble factors), or null
    const uint8_t *xflag;            // [item row][tile]: nonzero when some mask (extra time) of the row is
    int64_t mstride;
    const unsigned *stable;          // non-null: skip the pass when *stable (every scenario at its fixed point)
    int64_t *start, *finish;         // [op][scen]
    unsigned long long *arrive;      // [counted coll][scen] latest member launch
    unsigned *count;                 // [counted coll][tile] members arrived
    int64_t *slots;                  // [slot][scen] launch time of a slot collective's member, -1 before it
    int64_t *step;                   // [scen]
    uint64_t *digest;                // [scen] or null
    unsigned *status;
    int64_t spin_limit;              // wall-clock ticks (100 MHz) before a wait gives up
    int32_t n_scen, n_tiles;
    int32_t tile0, tiles;            // tiles handled by this launch
    int32_t n_walkers;
    int32_t final_pass;              // accumulate step time (and digest)
    int32_t store_all;               // store every start and finish (else only kNeedS / kNeedF)
    int32_t flag_rows;               // final mask pass: the variant that fetches only flagged rows (kInMaskFlags)
};


struct OverlapArgs {
    const int64_t *cl_off, *cp_off;
    const int32_t *cl;
    const uint8_t *cl_type;
    const ComputeRec *cp;
    const echo_scenario *scen;
    const int64_t *start, *finish;
    // rows of the walk items (cp_pos), mstride columns, as the walk reads them
    uint8_t *tmask;                  // in: masks of the previous pass (if it was refined), out: new ones
    uint32_t *ext;                   // prorating: in/out like tmask, the extra time q16(o, F) - o
    uint8_t *xflag;                  // out, [item row][tile]: nonzero when some mask (extra time) of the row is
    const int32_t *cp_pos;
    int64_t mstride;
    unsigned *chg;                   // non-null: [scen] set when some duration changes
    const unsigned *stable;          // non-null: skip when *stable
    // ensemble factors (forest_nodes non-null): features of the overlapping comm ops
    const int32_t *cl_coll;
    const int64_t *coll_bytes;       // S of each collective
    const int32_t *coll_N;           // N its cost uses
    const DevTreeNode *forest_nodes;
    const int32_t *forest_leaf;
    const int32_t *forest_roots;
    const int64_t *class_metrics;
    int32_t n_trees, forest_base;
    CompactForest fx;                // n_words > 0: the compact ensemble (LDS variant)
    int32_t prorate;                 // inflate only the overlapped part (extra times in ext)
    int32_t n_scen, n_tiles, n_ranks;
    int32_t prev_refined;            // the previous pass inflated its compute ops
    int32_t max_comm_streams;        // the most streams with comm ops on one rank (kernel variant)
    unsigned *status;
};

// Kernel launchers (echo_kernels.hip).  All enqueue on `stream`.
hipError_t launch_init(const DeviceGraph &g, const echo_scenario *scen, int32_t n_scen,
                       unsigned long long *arrive, int64_t n_arrive, unsigned *count,
                       int64_t n_count, int64_t *slots, int64_t n_slot_values, int64_t *step,
                       uint64_t *digest, hipStream_t stream);
hipError_t launch_clear(unsigned long long *arrive, int64_t n_arrive, unsigned *count,
                        int64_t n_count, int64_t *slots, int64_t n_slot_values, hipStream_t stream);
hipError_t launch_cc_cost(const CollTable &t, const echo_cc_table *tables, const echo_scenario *scen,
                          int32_t n_scen, int64_t *cost, unsigned *status, hipStream_t stream);
hipError_t launch_walk(const WalkArgs &a, int32_t n_blocks, hipStream_t stream);
hipError_t launch_overlap(const OverlapArgs &a, int32_t n_ranks, hipStream_t stream);
// Bins of the compact ensemble's per-collective (S, N) and per-compute-record (base
// duration) features.
hipError_t launch_forest_bins(const DeviceGraph &g, int64_t n_compute, const CompactForest &fx,
                              hipStream_t stream);
// After an overlap pass: count the refinement of every scenario whose durations changed,
// clear the change flags, and set *stable when none changed.
hipError_t launch_settle(unsigned *chg, int32_t n_scen, int32_t *refinements, unsigned *stable,
                         hipStream_t stream);
// Fill n int32 with v (a kernel, so the sequence stays capturable).
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream);
// Per-item input of a walk pass, the walk kernel's first template argument.
constexpr int kInNone = 0;        // first pass: base durations only
constexpr int kInMasks = 1;       // overlap masks, every row, fetched a round ahead into registers
constexpr int kInMaskFlags = 2;   // overlap masks, only flagged rows, staged in LDS (final passes)
constexpr int kInExtFlags = 3;    // prorated extra times, only flagged rows, staged in LDS
inline int walk_input(bool refined, bool prorate, bool flag_rows) {
    return !refined ? kInNone : prorate ? kInExtFlags : flag_rows ? kInMaskFlags : kInMasks;
}
// Co-resident walk workgroups (kBlockWalkers wavefronts each) the device can hold,
// for each kernel variant (bits 0-1 input, bit 2 final, bit 3 digest).
constexpr int kWalkVariants = 16;
hipError_t walk_capacity(int device, int64_t workgroups[kWalkVariants]);
inline int walk_variant(int in, bool final_pass, bool digest) {
    return in | (final_pass ? 4 : 0) | (digest ? 8 : 0);
}
// Device address of this GPU's fixed workspace array (ECHO_SCRATCH_BYTES) for
// echo_compose_batch_static; `device` must be current.  Looked up once per device.
hipError_t scratch_buffer(int device, void **ptr);
// Largest prorated extra time an op may carry (its staging slot is 32 bits).
constexpr uint32_t kExtLimit = 0xFFFFFFFFu;

}  // namespace echo
