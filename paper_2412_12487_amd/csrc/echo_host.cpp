// echo_host.cpp -- graph loader and C ABI of libecho.so.
//
// echo_load_graph is the simulator's initialisation step (Table 8 "Init."):
// it validates the per-rank graphs, matches collectives (Sec. 4.2 matching
// rules), merges every collective into one barrier node, levels the merged
// graph with Kahn's algorithm (a cycle is a deadlocked job), and lays out one
// level-ordered walk list per walker (a group of consecutive ranks walked by one
// wavefront) for the device.  echo_compose_batch is the
// execution step: it only enqueues kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <array>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "echo.h"
#include "echo_internal.h"

using namespace echo;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(ECHO_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int64_t kDurLimit = int64_t(1) << 43;
constexpr int64_t kBytesLimit = int64_t(1) << 50;
constexpr int64_t kI32Max = INT32_MAX;
constexpr int kMaxRanksPerWalker = 16;
constexpr int64_t kKnobLimitHost = int64_t(1) << 40;
constexpr int64_t kDefaultSpinNs = 20LL * 1000 * 1000 * 1000;   // 20 s
constexpr int64_t kMaxDevTreeNodes = int64_t(1) << 26;          // device ensemble: 1 GiB

// Table 6 (all-reduce breakdown): NCCL chunk size by tensor size.  The size
// row is read as MiB upper bounds, the chunk row in units of 1000 bytes.
int64_t table6_chunk(int64_t S) {
    static const int64_t kBound[] = {4, 8, 16, 32, 64, 128};
    static const int64_t kChunk[] = {18000, 36000, 72000, 72000, 72000, 144000};
    for (int i = 0; i < 6; ++i)
        if (S <= kBound[i] << 20) return kChunk[i];
    return 288000;
}

// Host side of a CollTable: the per-collective inputs of the CC model.
struct HostCollTable {
    int64_t n;
    std::vector<int64_t> bytes, chunk, eta_ring, eta_chunks;
    std::vector<int32_t> N, M, K;
    std::vector<uint8_t> type;
    explicit HostCollTable(int64_t count)
        : n(count), bytes(count), chunk(count), eta_ring(count), eta_chunks(count), N(count), M(count), K(count),
          type(count) {}
    void set(int64_t i, int t, int64_t S, int32_t members, int32_t servers, int32_t per_server) {
        const int64_t ch = table6_chunk(S);
        type[i] = (uint8_t)t;
        bytes[i] = S;
        chunk[i] = ch;
        eta_ring[i] = (S + (int64_t)members * ch - 1) / ((int64_t)members * ch);   // ring rounds
        eta_chunks[i] = (S + ch - 1) / ch;                                       // pipelined chunks
        N[i] = members;
        M[i] = servers;
        K[i] = per_server;
    }
};

template <class T>
hipError_t upload(T **dst, const std::vector<T> &src) {
    *dst = nullptr;
    const size_t bytes = std::max<size_t>(src.size(), 1) * sizeof(T);
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), bytes);
    if (e != hipSuccess) return e;
    if (!src.empty()) e = hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
    return e;
}

}  // namespace

struct echo_graph_s {
    int device = 0;
    int64_t n_ops = 0, n_colls = 0, n_levels = 0;
    int64_t n_items = 0;               // entries of the walk lists
    int64_t n_compute = 0;             // compute ops (overlap detection's compute records)
    int32_t n_ranks = 0, n_walkers = 0;
    int64_t capacity[kWalkVariants] = {};   // co-resident walk workgroups per kernel variant
    int64_t spin_limit = kDefaultSpinNs / 10;   // 100 MHz ticks
    int64_t max_launch_tiles = 0;      // > 0: at most this many scenario tiles per walk launch
    void *scratch = nullptr;           // this GPU's fixed workspace array (echo_compose_batch_static)
    hipError_t scratch_error = hipSuccess;
    DeviceGraph dg;
    std::vector<int32_t> counted_coll; // collective of each index among those met by counting
    std::vector<void *> owned;         // device allocations of the graph
    // workspace, grown on demand
    int64_t *class_cost = nullptr;
    size_t class_cost_n = 0;
    unsigned long long *arrive = nullptr;
    size_t arrive_n = 0;
    unsigned *count = nullptr;
    size_t count_n = 0;
    int64_t *slots = nullptr;
    size_t slots_n = 0;
    uint8_t *tmask = nullptr;
    size_t tmask_n = 0;
    uint32_t *ext = nullptr;           // prorated extra times
    size_t ext_n = 0;
    unsigned *chg = nullptr;           // per-scenario change flags + 1 stability word
    size_t chg_n = 0;
    int64_t *tmp_start = nullptr, *tmp_finish = nullptr;
    size_t tmp_start_n = 0, tmp_finish_n = 0;
    int64_t *tmp_step = nullptr;
    size_t tmp_step_n = 0;
    // optional kernel timing: (kind, start event, end event) per launch of the last compose
    bool timing = false;
    std::vector<hipEvent_t> events;
    std::vector<int32_t> timed_kinds;
};

namespace {

void free_compact(CompactForest &fx) {
    (void)hipFree(fx.words);
    (void)hipFree(fx.thr);
    (void)hipFree(fx.cbin);
    (void)hipFree(fx.coll_bin);
    (void)hipFree(fx.cp_bin);
    fx = CompactForest{};
}

void free_graph(echo_graph g) {
    if (!g) return;
    (void)hipSetDevice(g->device);
    (void)hipDeviceSynchronize();
    for (void *p : g->owned) (void)hipFree(p);
    (void)hipFree(g->class_cost);
    (void)hipFree(g->arrive);
    (void)hipFree(g->count);
    (void)hipFree(g->slots);
    (void)hipFree(g->tmask);
    (void)hipFree(g->dg.cc_tables);
    (void)hipFree(g->dg.forest_nodes);
    (void)hipFree(g->dg.forest_leaf);
    (void)hipFree(g->dg.forest_roots);
    (void)hipFree(g->dg.class_metrics);
    free_compact(g->dg.fx);
    (void)hipFree(g->ext);
    (void)hipFree(g->chg);
    (void)hipFree(g->tmp_start);
    (void)hipFree(g->tmp_finish);
    (void)hipFree(g->tmp_step);
    for (hipEvent_t ev : g->events) (void)hipEventDestroy(ev);
    delete g;
}

template <class T>
int ensure(T **p, size_t *have, size_t need, const char *what) {
    if (*have >= need && *p) return ECHO_OK;
    if (need > (size_t(1) << 56) / sizeof(T))        // far beyond any device; keeps the byte count exact
        return fail(ECHO_ERR_NOMEM, "workspace (%s): %zu elements", what, need);
    (void)hipFree(*p);
    *p = nullptr;
    *have = 0;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(p), std::max<size_t>(need, 1) * sizeof(T));
    if (e != hipSuccess) {
        *p = nullptr;
        return fail(ECHO_ERR_NOMEM, "workspace (%s, %zu bytes): %s", what, need * sizeof(T),
                    hipGetErrorString(e));
    }
    *have = need;
    return ECHO_OK;
}

// Bracket one kernel launch with events when timing is on.
struct Timed {
    echo_graph g;
    hipStream_t s;
    size_t slot = 0;
    hipError_t begin(int32_t kind) {
        if (!g->timing) return hipSuccess;
        slot = g->timed_kinds.size();
        while (g->events.size() < 2 * (slot + 1)) {
            hipEvent_t ev;
            hipError_t e = hipEventCreate(&ev);
            if (e != hipSuccess) return e;
            g->events.push_back(ev);
        }
        g->timed_kinds.push_back(kind);
        return hipEventRecord(g->events[2 * slot], s);
    }
    hipError_t end() { return g->timing ? hipEventRecord(g->events[2 * slot + 1], s) : hipSuccess; }
};

// ------------------------------------------------------------------ loader
int load(const echo_graph_desc *d, int device, int32_t min_rpw, echo_graph *out) {
    if (!d || !out) return fail(ECHO_ERR_ARG, "null descriptor or output handle");
    if (min_rpw < 0 || min_rpw > kMaxRanksPerWalker)
        return fail(ECHO_ERR_ARG, "ranks_per_walker %d outside [0, %d]", min_rpw, kMaxRanksPerWalker);
    *out = nullptr;
    const int64_t n = d->n_ops, nc = d->n_colls;
    const int64_t R = d->n_ranks;
    if (n < 0 || nc < 0 || R < 1 || d->gpus_per_node < 1)
        return fail(ECHO_ERR_ARG, "bad sizes: n_ops %lld, n_colls %lld, n_ranks %lld, gpus_per_node %d",
                    (long long)n, (long long)nc, (long long)R, d->gpus_per_node);
    if (n > kI32Max || nc > kI32Max) return fail(ECHO_ERR_RANGE, "more than 2^31 ops or collectives");
    if (!d->pred_off || (n > 0 && (!d->op_rank || !d->op_stream || !d->op_kind || !d->op_class ||
                                   !d->op_dur_ns || !d->op_coll)) ||
        (nc > 0 && (!d->coll_type || !d->coll_bytes)))
        return fail(ECHO_ERR_ARG, "null array in the graph descriptor");
    if (d->pred_off[0] != 0) return fail(ECHO_ERR_ARG, "pred_off[0] must be 0");
    if (d->pred_off[n] > kI32Max) return fail(ECHO_ERR_RANGE, "more than 2^31 explicit dependencies");
    if (d->pred_off[n] > 0 && !d->pred_idx) return fail(ECHO_ERR_ARG, "null pred_idx");

    // per-op checks
    for (int64_t v = 0; v < n; ++v) {
        const int32_t r = d->op_rank[v];
        if (r < 0 || r >= R || (v > 0 && r < d->op_rank[v - 1]))
            return fail(ECHO_ERR_ARG, "op %lld: rank %d out of range or not rank-major", (long long)v, r);
        if (d->op_stream[v] >= kStreams || d->op_kind[v] > ECHO_MEMCPY || d->op_class[v] >= kClasses)
            return fail(ECHO_ERR_ARG, "op %lld: bad stream/kind/class", (long long)v);
        if (d->op_kind[v] == ECHO_COMM) {
            if (d->op_coll[v] < 0 || d->op_coll[v] >= nc)
                return fail(ECHO_ERR_ARG, "comm op %lld names collective %lld", (long long)v,
                            (long long)d->op_coll[v]);
        } else {
            if (d->op_coll[v] != -1)
                return fail(ECHO_ERR_ARG, "non-comm op %lld names collective %lld", (long long)v,
                            (long long)d->op_coll[v]);
            if (d->op_dur_ns[v] < 0 || d->op_dur_ns[v] >= kDurLimit)
                return fail(ECHO_ERR_RANGE, "op %lld: duration %lld outside [0, 2^43)", (long long)v,
                            (long long)d->op_dur_ns[v]);
        }
        if (d->pred_off[v + 1] < d->pred_off[v])
            return fail(ECHO_ERR_ARG, "pred_off decreases at op %lld", (long long)v);
        for (int64_t j = d->pred_off[v]; j < d->pred_off[v + 1]; ++j) {
            const int64_t u = d->pred_idx[j];
            if (u < 0 || u >= v || d->op_rank[u] != r)
                return fail(ECHO_ERR_ARG, "op %lld depends on op %lld: must be an earlier op of its rank",
                            (long long)v, (long long)u);
        }
    }
    for (int64_t c = 0; c < nc; ++c) {
        if (d->coll_type[c] > ECHO_P2P) return fail(ECHO_ERR_ARG, "collective %lld: bad type", (long long)c);
        if (d->coll_bytes[c] < 0 || d->coll_bytes[c] >= kBytesLimit)
            return fail(ECHO_ERR_RANGE, "collective %lld: size outside [0, 2^50)", (long long)c);
    }

    // predecessors: previous op of the stream + explicit dependencies, deduplicated
    std::vector<int32_t> last(R * kStreams, -1);
    std::vector<int32_t> poff(n + 1, 0), preds;
    preds.reserve(n + d->pred_off[n]);
    {
        std::vector<int32_t> tmp;
        for (int64_t v = 0; v < n; ++v) {
            tmp.clear();
            const int64_t key = (int64_t)d->op_rank[v] * kStreams + d->op_stream[v];
            if (last[key] >= 0) tmp.push_back(last[key]);
            last[key] = (int32_t)v;
            for (int64_t j = d->pred_off[v]; j < d->pred_off[v + 1]; ++j) tmp.push_back(d->pred_idx[j]);
            std::sort(tmp.begin(), tmp.end());
            tmp.erase(std::unique(tmp.begin(), tmp.end()), tmp.end());
            preds.insert(preds.end(), tmp.begin(), tmp.end());
            if ((int64_t)preds.size() > kI32Max)
                return fail(ECHO_ERR_RANGE, "more than 2^31 merged dependencies");
            poff[v + 1] = (int32_t)preds.size();
        }
    }

    // collective membership: N, M (servers), K (most members on one server)
    std::vector<int64_t> moff(nc + 1, 0);
    for (int64_t v = 0; v < n; ++v)
        if (d->op_kind[v] == ECHO_COMM) ++moff[d->op_coll[v] + 1];
    for (int64_t c = 0; c < nc; ++c) moff[c + 1] += moff[c];
    std::vector<int32_t> mem(moff[nc]);
    {
        std::vector<int64_t> fill(moff.begin(), moff.end() - 1);
        for (int64_t v = 0; v < n; ++v)
            if (d->op_kind[v] == ECHO_COMM) mem[fill[d->op_coll[v]]++] = (int32_t)v;
    }
    const bool given = d->coll_N || d->coll_M || d->coll_K;
    if (given && !(d->coll_N && d->coll_M && d->coll_K))
        return fail(ECHO_ERR_ARG, "coll_N, coll_M and coll_K must be given together");
    std::vector<int32_t> cN(nc), cM(nc), cK(nc);   // members present, and the cost's N, M, K
    std::vector<int32_t> kN(nc), kM(nc), kK(nc);
    for (int64_t c = 0; c < nc; ++c) {
        const int64_t N = moff[c + 1] - moff[c];
        if (N == 0) return fail(ECHO_ERR_MATCH, "collective %lld has no member op", (long long)c);
        if (d->coll_type[c] == ECHO_P2P && N != 2)
            return fail(ECHO_ERR_MATCH, "P2P collective %lld has %lld members", (long long)c, (long long)N);
        int32_t servers = 0, best = 0, run = 0, prev_node = -1, prev_rank = -1;
        for (int64_t j = moff[c]; j < moff[c + 1]; ++j) {   // ascending op id => ascending rank
            const int32_t rk = d->op_rank[mem[j]];
            if (rk == prev_rank)
                return fail(ECHO_ERR_MATCH, "rank %d joins collective %lld twice", rk, (long long)c);
            prev_rank = rk;
            const int32_t node = rk / d->gpus_per_node;
            if (node != prev_node) {
                ++servers;
                run = 0;
                prev_node = node;
            }
            best = std::max(best, ++run);
        }
        cN[c] = (int32_t)N;
        cM[c] = servers;
        cK[c] = best;
        kN[c] = (int32_t)N;
        kM[c] = servers;
        kK[c] = best;
        if (given) {
            const int64_t gN = d->coll_N[c], gM = d->coll_M[c], gK = d->coll_K[c];
            if (gN < N || gM < 1 || gM > gN || gK < 1 || gK > gN || gM * gK < gN ||
                (d->coll_type[c] == ECHO_P2P && gN != 2))
                return fail(ECHO_ERR_ARG,
                            "collective %lld: membership N=%lld M=%lld K=%lld is inconsistent with its %lld "
                            "member op(s)", (long long)c, (long long)gN, (long long)gM, (long long)gK, (long long)N);
            kN[c] = (int32_t)gN;
            kM[c] = (int32_t)gM;
            kK[c] = (int32_t)gK;
        }
    }

    // matching rule: within one communicator (the (rank, stream) set of the
    // members) every member rank issues the communicator's collectives in the
    // same order -- so each collective sits at the same position everywhere.
    std::vector<int32_t> cid(nc);                  // communicator of each collective
    std::vector<int32_t> pos(nc, -1);              // its position in the communicator's issue order
    {
        std::map<std::vector<int64_t>, int32_t> comm_id;
        std::vector<int64_t> key;
        for (int64_t c = 0; c < nc; ++c) {
            key.clear();
            for (int64_t j = moff[c]; j < moff[c + 1]; ++j)
                key.push_back((int64_t)d->op_rank[mem[j]] * kStreams + d->op_stream[mem[j]]);
            auto it = comm_id.emplace(key, (int32_t)comm_id.size()).first;
            cid[c] = it->second;
        }
        std::unordered_map<uint64_t, int32_t> issued;   // (communicator, rank) -> collectives so far
        for (int64_t v = 0; v < n; ++v) {
            if (d->op_kind[v] != ECHO_COMM) continue;
            const int64_t c = d->op_coll[v];
            const uint64_t k = ((uint64_t)cid[c] << 32) | (uint32_t)d->op_rank[v];
            const int32_t p = issued[k]++;
            if (pos[c] < 0) pos[c] = p;
            else if (pos[c] != p)
                return fail(ECHO_ERR_MATCH,
                            "collective %lld: rank %d issues it as call %d of its communicator, "
                            "another member as call %d",
                            (long long)c, d->op_rank[v], p, pos[c]);
        }
    }

    // cost classes: collectives with the same (type, S, N, M, K) cost the same in every scenario
    std::vector<int32_t> ccls(nc);
    std::vector<std::array<int64_t, 5>> classes;
    {
        std::map<std::array<int64_t, 5>, int32_t> cls_id;
        for (int64_t c = 0; c < nc; ++c) {
            const std::array<int64_t, 5> k{d->coll_type[c], d->coll_bytes[c], kN[c], kM[c], kK[c]};
            auto it = cls_id.emplace(k, (int32_t)classes.size());
            if (it.second) classes.push_back(k);
            ccls[c] = it.first->second;
        }
    }
    // Kahn levels of the merged graph: node v for a compute/memcpy op,
    // node n + c for collective c (all its member ops).
    const int64_t nn = n + nc;
    auto node = [&](int64_t v) -> int64_t { return d->op_kind[v] == ECHO_COMM ? n + d->op_coll[v] : v; };
    std::vector<int64_t> soff(nn + 1, 0);
    std::vector<int32_t> indeg(nn, 0);
    for (int64_t v = 0; v < n; ++v)
        for (int32_t j = poff[v]; j < poff[v + 1]; ++j) {
            ++soff[node(preds[j]) + 1];
            ++indeg[node(v)];
        }
    for (int64_t x = 0; x < nn; ++x) soff[x + 1] += soff[x];
    std::vector<int64_t> succ(soff[nn]);
    {
        std::vector<int64_t> fill(soff.begin(), soff.end() - 1);
        for (int64_t v = 0; v < n; ++v)
            for (int32_t j = poff[v]; j < poff[v + 1]; ++j) succ[fill[node(preds[j])]++] = node(v);
    }
    std::vector<int32_t> level(nn, 0);
    std::vector<int64_t> queue;
    queue.reserve(nn);
    for (int64_t x = 0; x < nn; ++x)
        if (indeg[x] == 0) queue.push_back(x);
    for (size_t h = 0; h < queue.size(); ++h) {
        const int64_t x = queue[h];
        for (int64_t j = soff[x]; j < soff[x + 1]; ++j) {
            const int64_t y = succ[j];
            level[y] = std::max(level[y], level[x] + 1);
            if (--indeg[y] == 0) queue.push_back(y);
        }
    }
    if ((int64_t)queue.size() != nn) {
        for (int64_t c = 0; c < nc; ++c)
            if (indeg[n + c] > 0)
                return fail(ECHO_ERR_CYCLE, "dependency cycle through collective %lld: the simulated job deadlocks",
                            (long long)c);
        return fail(ECHO_ERR_CYCLE, "dependency cycle: the simulated job deadlocks");
    }
    int64_t n_levels = 0;
    for (int64_t x = 0; x < nn; ++x) n_levels = std::max<int64_t>(n_levels, level[x] + 1);
    std::vector<int32_t>().swap(indeg);
    std::vector<int64_t>().swap(succ);
    std::vector<int64_t>().swap(soff);

    // walkers: every walk workgroup of a scenario tile must be co-resident, so a
    // graph with more ranks than the device holds wavefronts walks several
    // consecutive ranks per wavefront
    hipError_t e = hipSetDevice(device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    int64_t capacity[kWalkVariants];
    e = walk_capacity(device, capacity);
    if (e != hipSuccess) return hip_fail(e, "occupancy query");
    const int64_t least = *std::min_element(capacity, capacity + kWalkVariants);
    int64_t rpw = std::max<int64_t>(1, min_rpw);       // ranks per walker
    while (rpw <= kMaxRanksPerWalker &&
           ((R + rpw - 1) / rpw + kBlockWalkers - 1) / kBlockWalkers > least)
        ++rpw;
    if (rpw > kMaxRanksPerWalker)
        return fail(ECHO_ERR_RANGE, "%lld ranks do not fit %lld co-resident walk workgroups of %d wavefronts "
                    "at %d ranks per wavefront", (long long)R, (long long)least, kBlockWalkers, kMaxRanksPerWalker);
    const int64_t W = (R + rpw - 1) / rpw;             // walkers
    const int64_t rpb = rpw * kBlockWalkers;           // ranks per workgroup

    // rank blocks (the ranks of one workgroup): the most used classes of a block
    // get its LDS cost slots; collectives whose members all sit in one block meet
    // in that block's LDS
    const int64_t nblk = (W + kBlockWalkers - 1) / kBlockWalkers;
    std::vector<int32_t> block_class(nblk * kClassSlots, -1);
    std::vector<uint32_t> coll_aux(nc, 0);          // channel part of the aux word (local collectives)
    std::vector<uint8_t> op_slot(n, (uint8_t)kNoSlot);
    {
        std::vector<int64_t> first_op(nblk + 1, n);
        for (int64_t v = n - 1; v >= 0; --v) first_op[d->op_rank[v] / rpb] = v;
        for (int64_t b = nblk - 1; b >= 0; --b)
            if (first_op[b] > first_op[b + 1]) first_op[b] = first_op[b + 1];
        std::unordered_map<int32_t, int64_t> use;
        std::vector<std::pair<int64_t, int32_t>> order;
        for (int64_t b = 0; b < nblk; ++b) {
            use.clear();
            for (int64_t v = first_op[b]; v < first_op[b + 1]; ++v)
                if (d->op_kind[v] == ECHO_COMM) ++use[ccls[d->op_coll[v]]];
            order.clear();
            for (auto &kv : use) order.emplace_back(-kv.second, kv.first);
            std::sort(order.begin(), order.end());
            std::unordered_map<int32_t, int32_t> slot_of;
            for (int i = 0; i < kClassSlots && i < (int)order.size(); ++i) {
                block_class[b * kClassSlots + i] = order[i].second;
                slot_of[order[i].second] = i;
            }
            for (int64_t v = first_op[b]; v < first_op[b + 1]; ++v)
                if (d->op_kind[v] == ECHO_COMM) {
                    auto it = slot_of.find(ccls[d->op_coll[v]]);
                    if (it != slot_of.end()) op_slot[v] = (uint8_t)it->second;
                }
        }
        // channels: one per communicator of a block whose collectives are all local
        std::map<std::pair<int64_t, int32_t>, int32_t> channel;   // (block, communicator) -> channel
        std::vector<int32_t> used(nblk, 0);
        for (int64_t c = 0; c < nc; ++c) {
            const int64_t b0 = d->op_rank[mem[moff[c]]] / rpb;
            bool local = true;
            for (int64_t j = moff[c]; j < moff[c + 1]; ++j)
                local = local && d->op_rank[mem[j]] / rpb == b0;
            const int64_t expected = (int64_t)cN[c] * (pos[c] / 2 + 1);
            if (!local || expected >= (int64_t(1) << kExpectedBits)) continue;
            auto it = channel.find({b0, cid[c]});
            if (it == channel.end()) {
                if (used[b0] >= kChannels) continue;                 // out of channels: meet globally
                it = channel.emplace(std::make_pair(b0, cid[c]), used[b0]++).first;
            }
            coll_aux[c] = kAuxLocal | ((uint32_t)it->second << 1) | ((uint32_t)(pos[c] & 1) << 4) |
                          ((uint32_t)expected << 9);
        }
        // a communicator is local for all its collectives or none: drop channels whose
        // communicator also has a collective that could not be met locally
        std::map<std::pair<int64_t, int32_t>, bool> ok;
        for (int64_t c = 0; c < nc; ++c) {
            const int64_t b0 = d->op_rank[mem[moff[c]]] / rpb;
            auto it = channel.find({b0, cid[c]});
            if (it == channel.end()) continue;
            auto &flag = ok.emplace(std::make_pair(b0, cid[c]), true).first->second;
            if (!(coll_aux[c] & kAuxLocal)) flag = false;
        }
        for (int64_t c = 0; c < nc; ++c) {
            const int64_t b0 = d->op_rank[mem[moff[c]]] / rpb;
            auto it = ok.find({b0, cid[c]});
            if (it != ok.end() && !it->second) coll_aux[c] = 0;
        }
    }
    // collectives met in device memory with few members meet through per-member slots
    std::vector<int64_t> slot_base(nc, -1);
    std::vector<int32_t> op_member(n, -1);        // position of a comm op among its collective's members
    int64_t n_slots = 0;
    for (int64_t c = 0; c < nc; ++c) {
        for (int64_t j = moff[c]; j < moff[c + 1]; ++j) op_member[mem[j]] = (int32_t)(j - moff[c]);
        if ((coll_aux[c] & kAuxLocal) || cN[c] > kSlotMembers || n_slots + cN[c] > kI32Max) continue;
        coll_aux[c] = kAuxSlots | ((uint32_t)cN[c] << 9);
        slot_base[c] = n_slots;
        n_slots += cN[c];
    }
    // the rest meet by counting arrivals in device memory: they get indices of their own,
    // so that the arrival maxima and counts a compose clears cover them only
    std::vector<int32_t> counted(nc, -1), counted_coll, counted_N;
    for (int64_t c = 0; c < nc; ++c)
        if (!(coll_aux[c] & (kAuxLocal | kAuxSlots))) {
            counted[c] = (int32_t)counted_coll.size();
            counted_coll.push_back((int32_t)c);
            counted_N.push_back(cN[c]);
        }
    auto item_coll = [&](int64_t c) { return counted[c] >= 0 ? counted[c] : (int32_t)c; };

    // walk lists: each walker's ops by (key, rank, program order), key = level
    // for compute/memcpy, the launch level for a comm op
    std::vector<int32_t> key(n);
    for (int64_t v = 0; v < n; ++v) {
        if (d->op_kind[v] == ECHO_COMM) {
            int32_t k = 0;
            for (int32_t j = poff[v]; j < poff[v + 1]; ++j) k = std::max(k, level[node(preds[j])] + 1);
            key[v] = k;
        } else {
            key[v] = level[v];
        }
    }
    std::vector<int64_t> op_off(W + 1, 0);            // ops of walker w: [op_off[w], op_off[w + 1])
    for (int64_t v = 0; v < n; ++v) ++op_off[d->op_rank[v] / rpw + 1];
    for (int64_t w = 0; w < W; ++w) op_off[w + 1] += op_off[w];
    std::vector<int32_t> order(n);
    for (int64_t v = 0; v < n; ++v) order[v] = (int32_t)v;   // rank-major already
    for (int64_t w = 0; w < W; ++w)
        std::stable_sort(order.begin() + op_off[w], order.begin() + op_off[w + 1],
                         [&](int32_t x, int32_t y) { return key[x] < key[y]; });
    std::vector<WalkItem> items;
    items.reserve(n);
    std::vector<int64_t> walk_off(W + 1, 0);
    std::vector<int32_t> far;
    {
        const int npair = (int)(rpw * kStreams);       // (rank, stream) pairs of a walker
        std::vector<int32_t> latest(kStreams);
        std::vector<int64_t> busy(npair), total(npair);
        std::vector<int> slot(npair);
        std::vector<int32_t> first_succ(n, -1);         // walk position of a comm op's first successor
        std::vector<std::pair<int32_t, int32_t>> sched; // (position, comm op) of the resolve items
        auto pair_of = [&](int64_t v, int64_t r0) { return (int)((d->op_rank[v] - r0) * kStreams + d->op_stream[v]); };
        // resolve item of comm op v: its barrier wait and finish; sv = its register slot
        // (-1: none), fold: also raise slot 0 to that finish for the compute op that follows
        auto emit_resolve = [&](int32_t v, int sv, bool fold) {
            WalkItem it{};
            it.op = v;
            it.meta = (uint32_t)kResolve | ((uint32_t)(sv >= 0 ? sv : 0) << 2) | (sv < 0 ? kNoReg : 0u) |
                      (fold ? kFold : 0u);
            const int64_t c = d->op_coll[v];
            // the collective's first member slot (slot mode), else unused
            it.far_off = slot_base[c] >= 0 ? (int32_t)slot_base[c] : (int32_t)far.size();
            it.coll = item_coll(c);
            it.dur = ccls[c];    // the cost class its finish reads
            it.nfar = 0;
            it.aux = coll_aux[d->op_coll[v]] | ((uint32_t)op_slot[v] << 5);
            items.push_back(it);
        };
        for (int64_t w = 0; w < W; ++w) {
            const int64_t r0 = w * rpw, lo = op_off[w], hi = op_off[w + 1];
            // slot 0 = the pair with the most compute/memcpy ops; one rank per walker:
            // the other streams keep their order; several: the busiest pairs get slots
            std::fill(busy.begin(), busy.end(), 0);
            std::fill(total.begin(), total.end(), 0);
            for (int64_t i = lo; i < hi; ++i) {
                ++total[pair_of(i, r0)];
                if (d->op_kind[i] != ECHO_COMM) ++busy[pair_of(i, r0)];
            }
            const int top = int(std::max_element(busy.begin(), busy.end()) - busy.begin());
            if (rpw == 1) {
                for (int k = 0, next = 1; k < kStreams; ++k) slot[k] = k == top ? 0 : next++;
            } else {
                std::vector<int> rest;
                for (int k = 0; k < npair; ++k)
                    if (k != top && total[k] > 0) rest.push_back(k);
                std::stable_sort(rest.begin(), rest.end(), [&](int x, int y) { return total[x] > total[y]; });
                std::fill(slot.begin(), slot.end(), -1);
                slot[top] = 0;
                for (int k = 0; k < (int)rest.size(); ++k) slot[rest[k]] = k + 1 < kStreams ? k + 1 : -1;
            }
            // Every comm op is finished by a resolve item placed right before its first
            // successor in the walk (or at the walk's end): its barrier is waited for as
            // late as the walk allows, and every reader of its slot comes after.
            sched.clear();
            for (int64_t i = lo; i < hi; ++i) {
                const int32_t v = order[i];
                for (int32_t j = poff[v]; j < poff[v + 1]; ++j) {
                    const int32_t u = preds[j];
                    if (d->op_kind[u] == ECHO_COMM && first_succ[u] < 0) {
                        first_succ[u] = (int32_t)(i - lo);
                        sched.emplace_back((int32_t)(i - lo), u);
                    }
                }
            }
            for (int64_t i = lo; i < hi; ++i) {
                const int32_t v = order[i];
                if (d->op_kind[v] == ECHO_COMM && first_succ[v] < 0) sched.emplace_back((int32_t)(hi - lo), v);
            }
            std::stable_sort(sched.begin(), sched.end(),
                             [](const std::pair<int32_t, int32_t> &x, const std::pair<int32_t, int32_t> &y) {
                                 return x.first < y.first;
                             });
            size_t next_due = 0;
            std::fill(latest.begin(), latest.end(), -1);
            for (int64_t i = lo; i < hi; ++i) {
                const int32_t v = order[i];
                const int sv = slot[pair_of(v, r0)];
                size_t due_end = next_due;
                while (due_end < sched.size() && sched[due_end].first == i - lo) ++due_end;
                // a compute/memcpy op of slot 0 whose other predecessors are exactly the comm ops
                // resolved right before it: the resolve items raise slot 0 to their finishes and
                // the op becomes a fast one (start = slot 0)
                bool fold = due_end > next_due && d->op_kind[v] != ECHO_COMM && sv == 0;
                for (int32_t j = poff[v]; fold && j < poff[v + 1]; ++j) {
                    const int32_t u = preds[j];
                    fold = u == latest[0] || (d->op_kind[u] == ECHO_COMM && first_succ[u] == i - lo);
                }
                for (; next_due < due_end; ++next_due) {
                    const int32_t u = sched[next_due].second;
                    emit_resolve(u, slot[pair_of(u, r0)], fold);
                }
                unsigned mask = 0;
                const int64_t f0 = (int64_t)far.size();
                for (int32_t j = poff[v]; j < poff[v + 1]; ++j) {
                    const int32_t u = preds[j];
                    if (fold && u != latest[0]) continue;          // folded into slot 0
                    const int su = slot[pair_of(u, r0)];
                    if (su >= 0 && latest[su] == u) mask |= 1u << su;
                    else far.push_back(u);
                }
                if (sv >= 0) latest[sv] = v;
                const bool fast = d->op_kind[v] != ECHO_COMM && sv == 0 && (mask & ~1u) == 0 &&
                                  (int64_t)far.size() == f0;
                WalkItem it{};
                it.op = v;
                it.meta = (uint32_t)d->op_kind[v] | ((uint32_t)(sv >= 0 ? sv : 0) << 2) |
                          ((uint32_t)d->op_class[v] << 5) | (mask << 8) | (fast ? kFast : 0u) |
                          (sv < 0 ? kNoReg : 0u);
                it.nfar = (int32_t)((int64_t)far.size() - f0);
                it.far_off = (int32_t)f0;
                it.coll = d->op_kind[v] == ECHO_COMM ? item_coll(d->op_coll[v]) : -1;
                it.aux = d->op_kind[v] == ECHO_COMM
                             ? coll_aux[d->op_coll[v]] | ((uint32_t)op_slot[v] << 5)
                             : 0u;
                if (d->op_kind[v] == ECHO_COMM) {
                    const int64_t c = d->op_coll[v];
                    it.dur = slot_base[c] >= 0 ? slot_base[c] + op_member[v] : 0;   // this member's slot
                } else {
                    it.dur = d->op_dur_ns[v];
                }
                items.push_back(it);
            }
            while (next_due < sched.size()) {
                const int32_t u = sched[next_due++].second;
                emit_resolve(u, slot[pair_of(u, r0)], false);
            }
            walk_off[w + 1] = (int64_t)items.size();
        }
    }
    if ((int64_t)far.size() > kI32Max || (int64_t)items.size() > kI32Max)
        return fail(ECHO_ERR_RANGE, "walk lists exceed 2^31 entries");
    {
        // member slots: every slot is written by exactly one launch item, and every
        // resolve item reads its collective's slots only (the kernels index with them)
        std::vector<uint8_t> written(n_slots, 0);
        for (const WalkItem &it : items) {
            const uint32_t x = (uint32_t)it.aux;
            if ((x & kAuxLocal) || !(x & kAuxSlots)) continue;
            const int64_t c = it.coll, base = slot_base[c], N = aux_expected(x);
            if (base < 0 || N != cN[c])
                return fail(ECHO_ERR_ARG, "internal: collective %lld has an inconsistent slot layout", (long long)c);
            if (item_kind(it.meta) == kResolve) {
                if (it.far_off != base || base + N > n_slots)
                    return fail(ECHO_ERR_ARG, "internal: resolve item of op %d reads slots out of range", it.op);
            } else if (it.dur < base || it.dur >= base + N || written[it.dur]++) {
                return fail(ECHO_ERR_ARG, "internal: launch item of op %d writes a wrong slot", it.op);
            }
        }
        for (int64_t k = 0; k < n_slots; ++k)
            if (!written[k]) return fail(ECHO_ERR_ARG, "internal: member slot %lld is never written", (long long)k);
    }
    {
        // what a pass without caller-visible timelines must still store
        std::vector<uint32_t> need(n, 0);
        for (int32_t u : far) need[u] |= kNeedF;
        // the last op of every overlap-detection block of a (rank, stream) compute list
        std::vector<int32_t> n_compute(R * kStreams, 0), i_compute(R * kStreams, 0);
        for (int64_t v = 0; v < n; ++v)
            if (d->op_kind[v] == ECHO_COMPUTE) ++n_compute[(int64_t)d->op_rank[v] * kStreams + d->op_stream[v]];
        for (int64_t v = 0; v < n; ++v)
            if (d->op_kind[v] == ECHO_COMPUTE) {
                const int64_t k = (int64_t)d->op_rank[v] * kStreams + d->op_stream[v];
                const int32_t i = i_compute[k]++;
                if (i % kOverlapBlock == kOverlapBlock - 1 || i == n_compute[k] - 1) need[v] |= kNeedF;
            }
        std::vector<int32_t> prev_on_stream(R * kStreams, -1);
        for (int64_t v = 0; v < n; ++v) {
            const int64_t k = (int64_t)d->op_rank[v] * kStreams + d->op_stream[v];
            const int32_t prev = prev_on_stream[k];
            prev_on_stream[k] = (int32_t)v;
            if (d->op_kind[v] == ECHO_COMM) {
                need[v] |= kNeedS | kNeedF;
            } else if (d->op_kind[v] == ECHO_COMPUTE) {
                const bool chained = prev >= 0 && d->op_kind[prev] == ECHO_COMPUTE && poff[v + 1] - poff[v] == 1 &&
                                     preds[poff[v]] == prev;
                if (!chained) need[v] |= kNeedS;
            }
        }
        for (WalkItem &it : items)
            if (item_kind(it.meta) != kResolve) it.meta |= need[it.op];
    }

    // per (rank, stream) comm and compute op lists in program order
    std::vector<int64_t> cl_off(R * kStreams + 1, 0), cp_off(R * kStreams + 1, 0);
    for (int64_t v = 0; v < n; ++v) {
        const int64_t k = (int64_t)d->op_rank[v] * kStreams + d->op_stream[v];
        if (d->op_kind[v] == ECHO_COMM) ++cl_off[k + 1];
        else if (d->op_kind[v] == ECHO_COMPUTE) ++cp_off[k + 1];
    }
    for (int64_t k = 0; k < R * kStreams; ++k) {
        cl_off[k + 1] += cl_off[k];
        cp_off[k + 1] += cp_off[k];
    }
    int32_t max_comm_streams = 0;
    for (int64_t r = 0; r < R; ++r) {
        int32_t k = 0;
        for (int st = 0; st < kStreams; ++st) k += cl_off[r * kStreams + st + 1] > cl_off[r * kStreams + st];
        max_comm_streams = std::max(max_comm_streams, k);
    }
    std::vector<int32_t> cl(cl_off.back()), cl_coll(cl_off.back());
    std::vector<uint8_t> cl_type(cl_off.back());
    std::vector<ComputeRec> cp(cp_off.back());
    std::vector<int32_t> cp_pos(cp_off.back());
    {
        // overlap detection writes its per-op outputs where the walk reads them: at the
        // row of the op's item (resolve items aside, every op has exactly one)
        std::vector<int32_t> item_pos(n, -1);
        for (size_t i = 0; i < items.size(); ++i)
            if (item_kind(items[i].meta) != kResolve) item_pos[items[i].op] = (int32_t)i;
        std::vector<int64_t> fl(cl_off.begin(), cl_off.end() - 1), fp(cp_off.begin(), cp_off.end() - 1);
        std::vector<int32_t> prev_on_stream(R * kStreams, -1);
        for (int64_t v = 0; v < n; ++v) {
            const int64_t k = (int64_t)d->op_rank[v] * kStreams + d->op_stream[v];
            const int32_t prev = prev_on_stream[k];
            prev_on_stream[k] = (int32_t)v;
            if (d->op_kind[v] == ECHO_COMM) {
                cl_type[fl[k]] = d->coll_type[d->op_coll[v]];
                cl_coll[fl[k]] = (int32_t)d->op_coll[v];
                cl[fl[k]++] = (int32_t)v;
            } else if (d->op_kind[v] == ECHO_COMPUTE) {
                // chained: the only predecessor is the previous op of the stream, a compute op
                const bool chained = prev >= 0 && d->op_kind[prev] == ECHO_COMPUTE && poff[v + 1] - poff[v] == 1 &&
                                     preds[poff[v]] == prev;
                cp_pos[fp[k]] = item_pos[v];
                cp[fp[k]++] = ComputeRec{(int32_t)v, (uint32_t)d->op_class[v] | (chained ? kChained : 0u),
                                         d->op_dur_ns[v]};
            }
        }
    }
    HostCollTable colls(nc), cls((int64_t)classes.size());
    for (int64_t c = 0; c < nc; ++c) colls.set(c, d->coll_type[c], d->coll_bytes[c], kN[c], kM[c], kK[c]);
    for (size_t k = 0; k < classes.size(); ++k)
        cls.set((int64_t)k, (int)classes[k][0], classes[k][1], (int32_t)classes[k][2], (int32_t)classes[k][3],
                (int32_t)classes[k][4]);

    // upload
    echo_graph g = new (std::nothrow) echo_graph_s();
    if (!g) return fail(ECHO_ERR_NOMEM, "host allocation");
    g->device = device;
    g->n_ops = n;
    g->n_items = (int64_t)items.size();
    g->n_compute = (int64_t)cp.size();
    g->n_colls = nc;
    g->n_levels = n_levels;
    g->n_ranks = (int32_t)R;
    g->n_walkers = (int32_t)W;
    std::copy(capacity, capacity + kWalkVariants, g->capacity);
    // set-up of the allocation-free compose: the device address of this GPU's workspace
    // array, looked up once per device (the device is current)
    g->scratch_error = scratch_buffer(device, &g->scratch);
    DeviceGraph &dg = g->dg;
    dg.n_ops = n;
    dg.n_colls = nc;
    dg.n_ranks = (int32_t)R;
    dg.n_walkers = (int32_t)W;
    dg.n_blocks = (int32_t)nblk;
    dg.max_comm_streams = max_comm_streams;
    dg.n_slots = n_slots;
    dg.n_counted = (int64_t)counted_coll.size();
    g->counted_coll = std::move(counted_coll);
#define UP(dst, src)                                                        \
    do {                                                                    \
        e = upload(&dst, src);                                              \
        if (dst) g->owned.push_back(dst);                                   \
        if (e != hipSuccess) {                                              \
            free_graph(g);                                                  \
            return fail(e == hipErrorOutOfMemory ? ECHO_ERR_NOMEM : ECHO_ERR_HIP, \
                        "uploading " #src ": %s", hipGetErrorString(e));    \
        }                                                                   \
    } while (0)
    UP(dg.items, items);
    UP(dg.walk_off, walk_off);
    UP(dg.far, far);
    for (int t = 0; t < 2; ++t) {
        HostCollTable &h = t == 0 ? colls : cls;
        CollTable &dt = t == 0 ? dg.colls : dg.classes;
        dt.n = h.n;
        UP(dt.bytes, h.bytes);
        UP(dt.chunk, h.chunk);
        UP(dt.eta_ring, h.eta_ring);
        UP(dt.eta_chunks, h.eta_chunks);
        UP(dt.N, h.N);
        UP(dt.M, h.M);
        UP(dt.K, h.K);
        UP(dt.type, h.type);
    }
    UP(dg.members, cN);
    UP(dg.counted_members, counted_N);
    UP(dg.block_class, block_class);
    UP(dg.cl_off, cl_off);
    UP(dg.cl, cl);
    UP(dg.cl_type, cl_type);
    UP(dg.cl_coll, cl_coll);
    UP(dg.cp_off, cp_off);
    UP(dg.cp, cp);
    UP(dg.cp_pos, cp_pos);
    UP(dg.status, std::vector<unsigned>(1, 0u));
#undef UP
    *out = g;
    return ECHO_OK;
}

// Device workspace of one compose call (see ensure_workspace for the sizes).
struct Workspace {
    int64_t *class_cost = nullptr;         // [class][scen] collective cost of each cost class
    unsigned long long *arrive = nullptr;  // [coll][scen] latest member launch
    unsigned *count = nullptr;             // [coll][tile] members arrived
    int64_t *slots = nullptr;              // [slot][scen] member launch times (slot collectives)
    uint8_t *tmask = nullptr;              // [item + kBlock][mstride] overlap masks (refined passes)
    uint32_t *ext = nullptr;               // same rows: prorated / ensemble extra times
    uint8_t *xflag = nullptr;              // [row][tile]: the row has a nonzero mask or extra time
    unsigned *chg = nullptr;               // [scen] change flags + 1 stability word (until_stable)
    int64_t *start = nullptr, *finish = nullptr, *step = nullptr;   // timelines (caller's or workspace)
};

struct ComposeShape {
    int64_t ns = 0;
    int32_t n_tiles = 0;
    int64_t mstride = 0, mrows = 0;
    bool until_stable = false, prorate = false, forest = false, ext = false;
};

int check_compose(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, const echo_validator &val,
                  ComposeShape *sh) {
    if (!g || !d_scen) return fail(ECHO_ERR_ARG, "null graph or scenario array");
    const int32_t n_refine = val.max_refine;
    sh->until_stable = val.until_stable != 0 && n_refine > 0;
    sh->prorate = val.prorate != 0 && n_refine > 0;
    sh->forest = val.forest != 0 && n_refine > 0;
    sh->ext = sh->prorate || sh->forest;           // refined passes add per-op extra times
    if (sh->forest && g->dg.n_trees == 0)
        return fail(ECHO_ERR_ARG, "forest factors requested, but the graph has no ensemble");
    if (n_scen < 1 || n_refine < 0 || n_refine > 64)
        return fail(ECHO_ERR_ARG, "n_scen must be >= 1 and 0 <= n_refine <= 64 (got %d, %d)", n_scen, n_refine);
    sh->ns = n_scen;
    sh->n_tiles = (int32_t)((sh->ns + kLanes - 1) / kLanes);
    // per-item outputs of overlap detection: whole tiles of columns, and one round of
    // rows past the last item (the walk fetches a round's rows at once)
    sh->mstride = (int64_t)sh->n_tiles * kLanes;
    sh->mrows = g->n_items + kBlock;
    return ECHO_OK;
}

// Workspace grown on demand in the graph's own device allocations.
int ensure_workspace(echo_graph g, const ComposeShape &sh, int32_t n_refine, int64_t *d_start, int64_t *d_finish,
                     int64_t *d_step, Workspace *ws) {
    const int64_t ns = sh.ns;
    int rc;
    if ((rc = ensure(&g->class_cost, &g->class_cost_n, (size_t)(g->dg.classes.n * ns), "class cost"))) return rc;
    if ((rc = ensure(&g->arrive, &g->arrive_n, (size_t)(g->dg.n_counted * ns), "arrivals"))) return rc;
    if ((rc = ensure(&g->count, &g->count_n, (size_t)(g->dg.n_counted * sh.n_tiles), "arrival counts"))) return rc;
    if ((rc = ensure(&g->slots, &g->slots_n, (size_t)(g->dg.n_slots * ns), "member slots"))) return rc;
    // overlap masks, then one flag byte per (item row, tile): whether the row has a nonzero one
    if (n_refine > 0 && !sh.ext &&
        (rc = ensure(&g->tmask, &g->tmask_n, (size_t)(sh.mrows * (sh.mstride + sh.n_tiles)), "overlap masks")))
        return rc;
    // extra times, then one flag byte per (item row, tile): whether the row has a nonzero one
    if (sh.ext && (rc = ensure(&g->ext, &g->ext_n,
                               (size_t)(sh.mrows * sh.mstride + (sh.mrows * sh.n_tiles + 3) / 4), "extra times")))
        return rc;
    if (sh.until_stable && (rc = ensure(&g->chg, &g->chg_n, (size_t)(ns + 1), "change flags"))) return rc;
    if (!d_start && (rc = ensure(&g->tmp_start, &g->tmp_start_n, (size_t)(g->n_ops * ns), "start"))) return rc;
    if (!d_finish && (rc = ensure(&g->tmp_finish, &g->tmp_finish_n, (size_t)(g->n_ops * ns), "finish")))
        return rc;
    if (!d_step && (rc = ensure(&g->tmp_step, &g->tmp_step_n, (size_t)ns, "step"))) return rc;
    ws->class_cost = g->class_cost;
    ws->arrive = g->arrive;
    ws->count = g->count;
    ws->slots = g->slots;
    ws->tmask = n_refine > 0 && !sh.ext ? g->tmask : nullptr;
    ws->ext = sh.ext ? g->ext : nullptr;
    ws->xflag = sh.ext ? reinterpret_cast<uint8_t *>(g->ext + sh.mrows * sh.mstride)
                       : (ws->tmask ? ws->tmask + sh.mrows * sh.mstride : nullptr);
    ws->chg = sh.until_stable ? g->chg : nullptr;
    ws->start = d_start ? d_start : g->tmp_start;
    ws->finish = d_finish ? d_finish : g->tmp_finish;
    ws->step = d_step ? d_step : g->tmp_step;
    return ECHO_OK;
}

// Enqueue one compose: init, class costs, pass 1, then per refinement overlap
// detection (+ settle) and the refined pass.  `timed`: record kernel events.
int enqueue_compose(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, const echo_validator &val,
                    const ComposeShape &sh, const Workspace &ws, bool store_all, uint64_t *d_digest,
                    int32_t *d_refinements, hipStream_t stream, bool timed) {
    const int32_t n_refine = val.max_refine;
    const int64_t ns = sh.ns;
    const int32_t n_tiles = sh.n_tiles;
    const bool until_stable = sh.until_stable, prorate = sh.prorate, forest = sh.forest, ext = sh.ext;
    unsigned *stable = until_stable ? ws.chg + ns : nullptr;
    hipError_t e;
    const int64_t n_arrive = g->dg.n_counted * ns, n_count = g->dg.n_counted * n_tiles,
                  n_slot_values = g->dg.n_slots * ns;
    g->timed_kinds.clear();
    const bool timing = timed && g->timing;
    Timed tm{g, stream};
#define TIMED(kind, call, what)                                                \
    do {                                                                       \
        if (timing && (e = tm.begin(kind))) return hip_fail(e, "event");       \
        if ((e = (call))) return hip_fail(e, what);                            \
        if (timing && (e = tm.end())) return hip_fail(e, "event");             \
    } while (0)
    TIMED(ECHO_K_INIT, launch_init(g->dg, d_scen, n_scen, ws.arrive, n_arrive, ws.count, n_count, ws.slots,
                                   n_slot_values, ws.step, d_digest, stream), "init kernel");
    TIMED(ECHO_K_CC_COST, launch_cc_cost(g->dg.classes, g->dg.cc_tables, d_scen, n_scen, ws.class_cost,
                                         g->dg.status, stream), "cc_cost kernel");
    if (until_stable && (e = launch_fill_i32(reinterpret_cast<int32_t *>(ws.chg), ns + 1, 0, stream)))
        return hip_fail(e, "fill kernel");
    if (d_refinements && (e = launch_fill_i32(d_refinements, ns, until_stable ? 0 : n_refine, stream)))
        return hip_fail(e, "fill kernel");
    // extra-time row flags start clear; overlap detection only sets them
    if (ext && n_refine > 0 &&
        (e = launch_fill_i32(reinterpret_cast<int32_t *>(ws.xflag), (sh.mrows * sh.n_tiles + 3) / 4, 0, stream)))
        return hip_fail(e, "fill kernel");

    for (int32_t p = 0; p <= n_refine; ++p) {
        // tiles per walk launch: every rank block of a tile must be co-resident (a final mask
        // pass may run either mask variant, so both count)
        const bool fin = p == n_refine, mask_pass = p > 0 && !ext;
        int64_t cap = g->capacity[walk_variant(walk_input(p > 0, ext, false), fin, d_digest != nullptr)];
        if (fin && mask_pass)
            cap = std::min(cap, g->capacity[walk_variant(kInMaskFlags, true, d_digest != nullptr)]);
        int64_t per_launch = std::max<int64_t>(1, std::min<int64_t>(n_tiles, cap / g->dg.n_blocks));
        if (g->max_launch_tiles > 0) per_launch = std::min<int64_t>(per_launch, g->max_launch_tiles);
        // A final mask pass whose launches average at least kFlagRowTiles tiles writes enough
        // timelines per unit of its chain of items for the fetched bytes to count, and fetches
        // only the flagged mask rows; with fewer tiles per launch it is bound by the chain and
        // fetches whole rows (measured on the 1024-rank graph: three tiles in one launch gain
        // 1.35 ms, four 1.3 ms, two neither gain nor lose; one-tile 32-scenario graphs lose
        // 0.5-2 ms, the 8192-rank graph's one tile per launch 1.1 ms per launch).
        const int64_t n_launches = (n_tiles + per_launch - 1) / per_launch;
        const bool flag_rows = fin && n_tiles >= kFlagRowTiles * n_launches;
        if (p > 0) {
            OverlapArgs o{};
            o.cl_off = g->dg.cl_off;
            o.cp_off = g->dg.cp_off;
            o.cl = g->dg.cl;
            o.cl_type = g->dg.cl_type;
            o.cp = g->dg.cp;
            o.scen = d_scen;
            o.start = ws.start;
            o.finish = ws.finish;
            o.tmask = ext ? nullptr : ws.tmask;
            o.ext = ext ? ws.ext : nullptr;
            o.xflag = ws.xflag;
            o.cp_pos = g->dg.cp_pos;
            o.mstride = sh.mstride;
            o.chg = until_stable ? ws.chg : nullptr;
            o.stable = stable;
            if (forest) {
                o.cl_coll = g->dg.cl_coll;
                o.coll_bytes = g->dg.colls.bytes;
                o.coll_N = g->dg.colls.N;
                o.forest_nodes = g->dg.forest_nodes;
                o.forest_leaf = g->dg.forest_leaf;
                o.forest_roots = g->dg.forest_roots;
                o.class_metrics = g->dg.class_metrics;
                o.n_trees = g->dg.n_trees;
                o.forest_base = g->dg.forest_base;
                o.fx = g->dg.fx;
            }
            o.prorate = prorate;
            o.n_scen = n_scen;
            o.n_tiles = n_tiles;
            o.n_ranks = g->n_ranks;
            o.prev_refined = p > 1;
            o.max_comm_streams = g->dg.max_comm_streams;
            o.status = g->dg.status;
            TIMED(ECHO_K_OVERLAP, launch_overlap(o, g->n_ranks, stream), "overlap kernel");
            if (until_stable && (e = launch_settle(ws.chg, n_scen, d_refinements, stable, stream)))
                return hip_fail(e, "settle kernel");
            TIMED(ECHO_K_CLEAR, launch_clear(ws.arrive, n_arrive, ws.count, n_count, ws.slots, n_slot_values, stream),
                  "clear kernel");
        }
        for (int64_t t0 = 0; t0 < n_tiles; t0 += per_launch) {
            WalkArgs a;
            a.items = g->dg.items;
            a.walk_off = g->dg.walk_off;
            a.far = g->dg.far;
            a.c_N = g->dg.counted_members;
            a.block_class = g->dg.block_class;
            a.scen = d_scen;
            a.class_cost = ws.class_cost;
            a.tmask = p > 0 && !ext ? ws.tmask : nullptr;
            a.ext = p > 0 && ext ? ws.ext : nullptr;
            a.xflag = p > 0 ? ws.xflag : nullptr;
            a.mstride = sh.mstride;
            a.stable = p < n_refine ? stable : nullptr;     // the final pass always runs
            a.start = ws.start;
            a.finish = ws.finish;
            a.arrive = ws.arrive;
            a.count = ws.count;
            a.slots = ws.slots;
            a.step = ws.step;
            a.digest = d_digest;
            a.status = g->dg.status;
            a.spin_limit = g->spin_limit;
            a.n_scen = n_scen;
            a.n_tiles = n_tiles;
            a.tile0 = (int32_t)t0;
            a.tiles = (int32_t)std::min<int64_t>(per_launch, n_tiles - t0);
            a.n_walkers = g->n_walkers;
            a.final_pass = p == n_refine;
            a.store_all = p == n_refine && store_all;
            a.flag_rows = flag_rows;
            if (g->n_ranks == 0 || g->n_ops == 0) continue;
            TIMED(ECHO_K_WALK, launch_walk(a, g->dg.n_blocks, stream), "walk kernel");
        }
    }
#undef TIMED
    return ECHO_OK;
}

int compose(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, const echo_validator &val, int64_t *d_start,
            int64_t *d_finish, int64_t *d_step, uint64_t *d_digest, int32_t *d_refinements, hipStream_t stream) {
    ComposeShape sh;
    int rc = check_compose(g, d_scen, n_scen, val, &sh);
    if (rc) return rc;
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    Workspace ws;
    if ((rc = ensure_workspace(g, sh, val.max_refine, d_start, d_finish, d_step, &ws))) return rc;
    return enqueue_compose(g, d_scen, n_scen, val, sh, ws, d_start || d_finish, d_digest, d_refinements, stream,
                           true);
}

// Longest chain of the walk (echo_walk_chain): every walker's items run in list
// order; a resolve item also waits for the launch items of every member of its
// collective.  The walk lists drain in this order by construction (the loader's
// key order), so a walker only ever waits for launches that are still to come.
int walk_chain(echo_graph g, const int64_t w[3], int64_t out[4]) {
    struct Pt {
        int64_t len = 0, items = 0, loc = 0, glob = 0;
    };
    auto later = [](const Pt &a, const Pt &b) { return a.len > b.len ? a : b; };
    const int64_t W = g->n_walkers, nc = g->n_colls, n_items = g->n_items;
    std::vector<WalkItem> items(n_items);
    std::vector<int64_t> off(W + 1, 0);
    std::vector<int32_t> members(nc);
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    if (n_items > 0 && (e = hipMemcpy(items.data(), g->dg.items, n_items * sizeof(WalkItem), hipMemcpyDeviceToHost)))
        return hip_fail(e, "walk list download");
    if (W > 0 && (e = hipMemcpy(off.data(), g->dg.walk_off, (W + 1) * sizeof(int64_t), hipMemcpyDeviceToHost)))
        return hip_fail(e, "walk offsets download");
    if (nc > 0 && (e = hipMemcpy(members.data(), g->dg.members, nc * sizeof(int32_t), hipMemcpyDeviceToHost)))
        return hip_fail(e, "member counts download");
    std::vector<Pt> cur(W), cmax(nc);
    std::vector<int32_t> arrived(nc, 0), wait_head(nc, -1), wait_next(W, -1);
    std::vector<int64_t> pos(off.begin(), off.end() - (W > 0 ? 1 : 0));
    std::vector<int32_t> runnable;
    for (int64_t x = W - 1; x >= 0; --x) runnable.push_back((int32_t)x);
    int64_t done = 0;
    while (!runnable.empty()) {
        const int32_t x = runnable.back();
        runnable.pop_back();
        for (; pos[x] < off[x + 1]; ++pos[x]) {
            WalkItem it = items[pos[x]];
            const int kind = item_kind(it.meta);
            if ((kind == ECHO_COMM || kind == kResolve) && !((uint32_t)it.aux & (kAuxLocal | kAuxSlots))) {
                if (it.coll < 0 || it.coll >= (int32_t)g->counted_coll.size())
                    return fail(ECHO_ERR_ARG, "internal: walk item of op %d has no counted collective", it.op);
                it.coll = g->counted_coll[it.coll];
            }
            Pt p = cur[x];
            if (kind == kResolve) {
                if (arrived[it.coll] < members[it.coll]) {     // some member has not launched yet
                    wait_next[x] = wait_head[it.coll];
                    wait_head[it.coll] = x;
                    break;
                }
                p = later(p, cmax[it.coll]);
                const bool local = ((uint32_t)it.aux & kAuxLocal) != 0;
                p.len += w[0] + (local ? w[1] : w[2]);
                (local ? p.loc : p.glob) += 1;
            } else {
                p.len += w[0];
            }
            p.items += 1;
            cur[x] = p;
            ++done;
            if (kind == ECHO_COMM) {
                cmax[it.coll] = later(cmax[it.coll], p);
                if (++arrived[it.coll] == members[it.coll])
                    for (int32_t y = wait_head[it.coll]; y >= 0; y = wait_next[y]) runnable.push_back(y);
            }
        }
    }
    if (done != n_items) return fail(ECHO_ERR_ARG, "walk lists do not drain (%lld of %lld items)", (long long)done,
                                     (long long)n_items);
    Pt best;
    for (const Pt &p : cur) best = later(best, p);
    out[0] = best.len;
    out[1] = best.items;
    out[2] = best.loc;
    out[3] = best.glob;
    return ECHO_OK;
}

}  // namespace

extern "C" {

int echo_load_graph_ex(const echo_graph_desc *desc, int hip_device, int32_t ranks_per_walker, echo_graph *out) {
    g_last_error.clear();
    try {
        return load(desc, hip_device, ranks_per_walker, out);
    } catch (const std::bad_alloc &) {
        return fail(ECHO_ERR_NOMEM, "host allocation failed while loading the graph");
    } catch (...) {
        return fail(ECHO_ERR_ARG, "unexpected exception while loading the graph");
    }
}

int echo_load_graph(const echo_graph_desc *desc, int hip_device, echo_graph *out) {
    return echo_load_graph_ex(desc, hip_device, 0, out);
}

int echo_graph_info(echo_graph g, int64_t *n_ops, int64_t *n_colls, int64_t *n_levels) {
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    if (n_ops) *n_ops = g->n_ops;
    if (n_colls) *n_colls = g->n_colls;
    if (n_levels) *n_levels = g->n_levels;
    return ECHO_OK;
}

void echo_free_graph(echo_graph g) { free_graph(g); }

int echo_cc_cost(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int64_t *d_cost, void *hip_stream) {
    g_last_error.clear();
    if (!g || !d_scen || !d_cost || n_scen < 1) return fail(ECHO_ERR_ARG, "null argument or n_scen < 1");
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    if ((e = launch_init(g->dg, d_scen, n_scen, nullptr, 0, nullptr, 0, nullptr, 0, nullptr, nullptr, s)))
        return hip_fail(e, "init kernel");
    if ((e = launch_cc_cost(g->dg.colls, g->dg.cc_tables, d_scen, n_scen, d_cost, g->dg.status, s)))
        return hip_fail(e, "cc_cost kernel");
    return ECHO_OK;
}

int echo_compose_batch(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int32_t n_refine,
                       int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                       void *hip_stream) {
    g_last_error.clear();
    try {
        if (n_refine < 0 || n_refine > 64)
            return fail(ECHO_ERR_ARG, "n_refine must be in 0..64 (got %d)", n_refine);
        const echo_validator val{n_refine, 0, 0};
        return compose(g, d_scen, n_scen, val, d_start, d_finish, d_step, d_digest, nullptr,
                       static_cast<hipStream_t>(hip_stream));
    } catch (...) {
        return fail(ECHO_ERR_NOMEM, "unexpected exception in compose");
    }
}

int echo_compose_validated(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, const echo_validator *opts,
                           int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                           int32_t *d_refinements, void *hip_stream) {
    g_last_error.clear();
    try {
        if (!opts) return fail(ECHO_ERR_ARG, "null validator options");
        if (opts->max_refine < 0 || opts->max_refine > 64)
            return fail(ECHO_ERR_ARG, "max_refine must be in 0..64 (got %d)", opts->max_refine);
        return compose(g, d_scen, n_scen, *opts, d_start, d_finish, d_step, d_digest, d_refinements,
                       static_cast<hipStream_t>(hip_stream));
    } catch (...) {
        return fail(ECHO_ERR_NOMEM, "unexpected exception in compose");
    }
}

int echo_compose_batch_static(echo_graph g, const echo_scenario *d_scen, int32_t n_scen, int32_t n_refine,
                              int64_t *d_start, int64_t *d_finish, int64_t *d_step, uint64_t *d_digest,
                              void *hip_stream) {
    g_last_error.clear();
    try {
        if (n_refine < 0 || n_refine > 64)
            return fail(ECHO_ERR_ARG, "n_refine must be in 0..64 (got %d)", n_refine);
        if (!d_start || !d_finish || !d_step)
            return fail(ECHO_ERR_ARG, "the allocation-free compose needs d_start, d_finish and d_step");
        const echo_validator val{n_refine, 0, 0, 0};
        ComposeShape sh;
        int rc = check_compose(g, d_scen, n_scen, val, &sh);
        if (rc) return rc;
        if (!g->scratch)
            return hip_fail(g->scratch_error != hipSuccess ? g->scratch_error : hipErrorInvalidSymbol,
                            "workspace array of this GPU");
        // the workspace's parts, each rounded up to 256 bytes; sizes checked before any
        // product could exceed 64 bits (every factor is below 2^32)
        constexpr int64_t kCap = ECHO_SCRATCH_BYTES;
        const int64_t parts[5] = {
            g->dg.classes.n * sh.ns * (int64_t)sizeof(int64_t),              // class costs
            g->dg.n_counted * sh.ns * (int64_t)sizeof(unsigned long long),   // arrival maxima
            g->dg.n_counted * sh.n_tiles * (int64_t)sizeof(unsigned),         // arrival counts
            n_refine > 0 ? sh.mrows * (sh.mstride + sh.n_tiles) : 0,         // overlap masks and row flags
            g->dg.n_slots * sh.ns * (int64_t)sizeof(int64_t),               // member slots
        };
        int64_t offs[5], total = 0;
        for (int i = 0; i < 5; ++i) {
            offs[i] = total;
            if (parts[i] > kCap) {
                total = kCap + 1;
                break;
            }
            total += (parts[i] + 255) / 256 * 256;
        }
        if (total > kCap)
            return fail(ECHO_ERR_RANGE,
                        "the allocation-free compose needs more workspace than its fixed %lld-byte array "
                        "(%lld scenarios, %lld collectives, %lld walk items)",
                        (long long)kCap, (long long)sh.ns, (long long)g->n_colls, (long long)g->n_items);
        hipError_t e = hipSetDevice(g->device);
        if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
        uint8_t *const base = static_cast<uint8_t *>(g->scratch);
        Workspace ws;
        ws.class_cost = reinterpret_cast<int64_t *>(base + offs[0]);
        ws.arrive = reinterpret_cast<unsigned long long *>(base + offs[1]);
        ws.count = reinterpret_cast<unsigned *>(base + offs[2]);
        ws.tmask = n_refine > 0 ? base + offs[3] : nullptr;
        ws.xflag = n_refine > 0 ? base + offs[3] + sh.mrows * sh.mstride : nullptr;
        ws.slots = reinterpret_cast<int64_t *>(base + offs[4]);
        ws.start = d_start;
        ws.finish = d_finish;
        ws.step = d_step;
        // init clears the arrival maxima, counts and member slots; every mask a refined pass reads is
        // written by the overlap detection before it, and class costs by the CC kernel
        return enqueue_compose(g, d_scen, n_scen, val, sh, ws, true, d_digest, nullptr,
                               static_cast<hipStream_t>(hip_stream), false);
    } catch (...) {
        return fail(ECHO_ERR_NOMEM, "unexpected exception in compose");
    }
}

int echo_set_cc_tables(echo_graph g, const echo_cc_table *tables, int32_t n_tables) {
    g_last_error.clear();
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    if (n_tables < 0 || (n_tables > 0 && !tables)) return fail(ECHO_ERR_ARG, "bad table array (n_tables %d)", n_tables);
    constexpr int64_t kLim = kKnobLimitHost;
    for (int32_t k = 0; k < n_tables; ++k) {
        const echo_cc_table &t = tables[k];
        for (int i = 0; i < ECHO_CC_ROWS; ++i) {
            if (i > 0 && t.max_bytes[i] < t.max_bytes[i - 1])
                return fail(ECHO_ERR_ARG, "table %d: max_bytes decreases at row %d", k, i);
            if (t.chunk[i] < 1 || t.chunk[i] >= (int64_t(1) << 32) || t.alpha_ns[i] < 0 || t.alpha_ns[i] >= kLim ||
                t.beta_ns[i] < 0 || t.beta_ns[i] >= kLim || t.gamma_ns[i] < 0 || t.gamma_ns[i] >= kLim ||
                t.reduce_MBps[i] < 1 || t.reduce_MBps[i] >= kLim)
                return fail(ECHO_ERR_RANGE, "table %d row %d: value out of range", k, i);
        }
    }
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    echo_cc_table *d = nullptr;
    if (n_tables > 0) {
        e = hipMalloc(reinterpret_cast<void **>(&d), sizeof(echo_cc_table) * (size_t)n_tables);
        if (e != hipSuccess) return fail(ECHO_ERR_NOMEM, "CC tables: %s", hipGetErrorString(e));
        e = hipMemcpy(d, tables, sizeof(echo_cc_table) * (size_t)n_tables, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(d);
            return hip_fail(e, "CC tables upload");
        }
    }
    // composes already enqueued may still read the old tables
    (void)hipDeviceSynchronize();
    (void)hipFree(g->dg.cc_tables);
    g->dg.cc_tables = d;
    g->dg.n_cc_tables = n_tables;
    return ECHO_OK;
}

static int set_forest(echo_graph g, const echo_tree_node *nodes, int64_t n_nodes, const int32_t *roots,
                      int32_t n_trees, int32_t base_q16, const int64_t *class_metrics) {
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    if (n_trees < 0) return fail(ECHO_ERR_ARG, "n_trees %d < 0", n_trees);
    if (n_trees > 0) {
        if (!nodes || !roots || !class_metrics || n_nodes < 1 || n_nodes > kI32Max)
            return fail(ECHO_ERR_ARG, "null or empty ensemble arrays");
        if (base_q16 < 65536 || base_q16 >= (1 << 20)) return fail(ECHO_ERR_ARG, "base %d outside [65536, 2^20)", base_q16);
        // every path at most ECHO_TREE_DEPTH splits, indices and features in range
        std::vector<std::pair<int32_t, int32_t>> stack;
        for (int32_t t = 0; t < n_trees; ++t) {
            if (roots[t] < 0 || roots[t] >= n_nodes) return fail(ECHO_ERR_ARG, "tree %d: root out of range", t);
            stack.assign(1, {roots[t], 0});
            while (!stack.empty()) {
                const auto [i, depth] = stack.back();
                stack.pop_back();
                const echo_tree_node &nd = nodes[i];
                if (nd.feature < 0) continue;
                if (depth >= ECHO_TREE_DEPTH || nd.feature >= 12 || nd.left < 0 || nd.left >= n_nodes || nd.right < 0 ||
                    nd.right >= n_nodes)
                    return fail(ECHO_ERR_ARG, "tree %d: node %d is malformed or deeper than %d", t, i, ECHO_TREE_DEPTH);
                stack.push_back({nd.left, depth + 1});
                stack.push_back({nd.right, depth + 1});
            }
        }
    }
    // device layout: each tree laid out breadth first from its root, a split's two
    // children side by side (a node reached along two paths is copied)
    std::vector<DevTreeNode> hn;
    std::vector<int32_t> hleaf;
    std::vector<uint8_t> is_leaf;
    std::vector<int32_t> hr(n_trees);
    std::vector<std::pair<int32_t, int64_t>> todo;    // (source node, device slot)
    for (int32_t t = 0; t < n_trees; ++t) {
        hr[t] = (int32_t)hn.size();
        hn.push_back(DevTreeNode{});
        todo.assign(1, {roots[t], (int64_t)hr[t]});
        for (size_t h = 0; h < todo.size(); ++h) {
            const echo_tree_node &nd = nodes[todo[h].first];
            const int64_t slot = todo[h].second;
            if (nd.feature < 0) {
                hn[slot] = DevTreeNode{INT64_MIN, 0, (int32_t)slot - 1};   // loops to itself
                hleaf.resize(hn.size());
                hleaf[slot] = nd.value;
                is_leaf.resize(hn.size());
                is_leaf[slot] = 1;
                continue;
            }
            if ((int64_t)hn.size() + 2 > kMaxDevTreeNodes)
                return fail(ECHO_ERR_RANGE, "ensemble too large: more than %lld nodes once laid out",
                            (long long)kMaxDevTreeNodes);
            const int32_t l = (int32_t)hn.size();
            hn.push_back(DevTreeNode{});
            hn.push_back(DevTreeNode{});
            hn[slot] = DevTreeNode{nd.threshold, nd.feature, l};
            todo.push_back({nd.left, (int64_t)l});
            todo.push_back({nd.right, (int64_t)l + 1});
        }
    }
    hleaf.resize(hn.size());
    is_leaf.resize(hn.size());
    // compact form (overlap detection keeps it in LDS): thresholds ranked per feature,
    // one 32-bit word per node; left out when a limit of the word layout or of the LDS
    // budget is exceeded (the ensemble is then walked from device memory)
    std::vector<uint32_t> words;
    std::vector<int64_t> thr;
    int32_t thr_off[kFxFeatures + 1] = {};
    std::vector<int32_t> cbin;
    int32_t tbin[4] = {};
    if (n_trees > 0 && (int64_t)hn.size() + n_trees <= kFxMaxWords) {
        std::vector<std::vector<int64_t>> tf(kFxFeatures);
        for (size_t i = 0; i < hn.size(); ++i)
            if (!is_leaf[i]) tf[hn[i].feature].push_back(hn[i].threshold);
        bool fits = true;
        for (int f = 0; f < kFxFeatures; ++f) {
            std::sort(tf[f].begin(), tf[f].end());
            tf[f].erase(std::unique(tf[f].begin(), tf[f].end()), tf[f].end());
            fits = fits && (int64_t)tf[f].size() < (int64_t(1) << kFxRankBits);
            thr_off[f + 1] = thr_off[f] + (int32_t)tf[f].size();
            thr.insert(thr.end(), tf[f].begin(), tf[f].end());
        }
        // bin of x for feature f: thresholds <= x
        auto bin = [&](int f, int64_t x) {
            return (int32_t)(std::upper_bound(tf[f].begin(), tf[f].end(), x) - tf[f].begin());
        };
        for (size_t i = 0; fits && i < hn.size(); ++i) {
            if (is_leaf[i]) {
                const int64_t v = hleaf[i];
                fits = v >= -(int64_t(1) << 27) && v < (int64_t(1) << 27);
                words.push_back((uint32_t)(int32_t)(v * 16) | kFxLeaf);
            } else {
                const int f = hn[i].feature;
                const int64_t r = std::lower_bound(tf[f].begin(), tf[f].end(), hn[i].threshold) - tf[f].begin();
                const int64_t off = (int64_t)hn[i].left - (int64_t)i;
                fits = off >= 1 && off < (int64_t(1) << (32 - 4 - kFxRankBits));
                words.push_back((uint32_t)f | ((uint32_t)r << 4) | ((uint32_t)off << (4 + kFxRankBits)));
            }
        }
        if (fits) {
            cbin.assign(kClasses * kFxFeatures, 0);
            for (int k = 0; k < kClasses; ++k) {
                cbin[k * kFxFeatures + 0] = bin(0, k);
                for (int j = 0; j < kClassMetrics; ++j)
                    cbin[k * kFxFeatures + 8 + j] = bin(8 + j, class_metrics[k * kClassMetrics + j]);
            }
            for (int t = 0; t < 4; ++t) tbin[t] = bin(2, t);
        } else {
            words.clear();
        }
    }
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    (void)hipDeviceSynchronize();                  // composes already enqueued may read the old ensemble
    (void)hipFree(g->dg.forest_nodes);
    (void)hipFree(g->dg.forest_leaf);
    (void)hipFree(g->dg.forest_roots);
    (void)hipFree(g->dg.class_metrics);
    free_compact(g->dg.fx);
    g->dg.forest_nodes = nullptr;
    g->dg.forest_leaf = nullptr;
    g->dg.forest_roots = nullptr;
    g->dg.class_metrics = nullptr;
    g->dg.n_trees = 0;
    if (n_trees == 0) return ECHO_OK;
    std::vector<int64_t> hm(class_metrics, class_metrics + kClasses * kClassMetrics);
    auto nomem = [&](hipError_t err) {
        return fail(err == hipErrorOutOfMemory ? ECHO_ERR_NOMEM : ECHO_ERR_HIP, "ensemble upload: %s",
                    hipGetErrorString(err));
    };
    if ((e = upload(&g->dg.forest_nodes, hn)) || (e = upload(&g->dg.forest_leaf, hleaf)) ||
        (e = upload(&g->dg.forest_roots, hr)) ||
        (e = upload(&g->dg.class_metrics, hm)))
        return nomem(e);
    if (!words.empty()) {
        CompactForest &fx = g->dg.fx;
        std::copy(thr_off, thr_off + kFxFeatures + 1, fx.thr_off);
        std::copy(tbin, tbin + 4, fx.tbin);
        if ((e = upload(&fx.words, words)) || (e = upload(&fx.thr, thr)) || (e = upload(&fx.cbin, cbin)) ||
            (e = hipMalloc(reinterpret_cast<void **>(&fx.coll_bin), sizeof(int32_t) * 2 * std::max<int64_t>(g->n_colls, 1))) ||
            (e = hipMalloc(reinterpret_cast<void **>(&fx.cp_bin),
                           sizeof(int32_t) * std::max<int64_t>(g->n_compute, 1)))) {
            free_compact(fx);
            return nomem(e);
        }
        // per-collective and per-compute-record bins, computed on the device where the
        // graph's sizes and durations live
        if ((e = launch_forest_bins(g->dg, g->n_compute, fx, nullptr)) || (e = hipDeviceSynchronize())) {
            free_compact(fx);
            return hip_fail(e, "ensemble bins");
        }
        fx.n_words = (int32_t)words.size();
    }
    g->dg.n_trees = n_trees;
    g->dg.forest_base = base_q16;
    return ECHO_OK;
}

int echo_set_forest(echo_graph g, const echo_tree_node *nodes, int64_t n_nodes, const int32_t *roots,
                    int32_t n_trees, int32_t base_q16, const int64_t *class_metrics) {
    g_last_error.clear();
    try {
        return set_forest(g, nodes, n_nodes, roots, n_trees, base_q16, class_metrics);
    } catch (const std::bad_alloc &) {
        return fail(ECHO_ERR_NOMEM, "host allocation failed while laying out the ensemble");
    } catch (...) {
        return fail(ECHO_ERR_ARG, "unexpected exception while setting the ensemble");
    }
}

int echo_sync_status(echo_graph g, void *hip_stream) {
    g_last_error.clear();
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    if ((e = hipStreamSynchronize(static_cast<hipStream_t>(hip_stream)))) return hip_fail(e, "stream sync");
    unsigned st = 0;
    if ((e = hipMemcpy(&st, g->dg.status, sizeof st, hipMemcpyDeviceToHost))) return hip_fail(e, "status read");
    const unsigned zero = 0;
    if ((e = hipMemcpy(g->dg.status, &zero, sizeof zero, hipMemcpyHostToDevice))) return hip_fail(e, "status clear");
    if (st & kStatusTimeout)
        return fail(ECHO_ERR_DEVICE, "a collective barrier wait exceeded the spin limit");
    if (st & kStatusRange) return fail(ECHO_ERR_RANGE, "a scenario knob is out of range");
    if (st & kStatusOverflow) return fail(ECHO_ERR_RANGE, "a time reached 2^62 ns");
    return ECHO_OK;
}

int echo_set_timing(echo_graph g, int enable) {
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    g->timing = enable != 0;
    g->timed_kinds.clear();
    return ECHO_OK;
}

int echo_kernel_times(echo_graph g, int32_t max, int32_t *kinds, float *ms, int32_t *n) {
    g_last_error.clear();
    if (!g || !n || max < 0 || (max > 0 && (!kinds || !ms))) return fail(ECHO_ERR_ARG, "null argument");
    const int32_t k = (int32_t)g->timed_kinds.size();
    *n = k;
    hipError_t e = hipSetDevice(g->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    for (int32_t i = 0; i < k && i < max; ++i) {
        kinds[i] = g->timed_kinds[i];
        if ((e = hipEventElapsedTime(&ms[i], g->events[2 * i], g->events[2 * i + 1])))
            return hip_fail(e, "hipEventElapsedTime");
    }
    return ECHO_OK;
}

int echo_set_spin_limit(echo_graph g, int64_t limit_ns) {
    g_last_error.clear();
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    if (limit_ns < 10 || limit_ns > (int64_t(1) << 40))
        return fail(ECHO_ERR_ARG, "spin limit %lld ns outside [10, 2^40]", (long long)limit_ns);
    g->spin_limit = limit_ns / 10;
    return ECHO_OK;
}

int echo_set_launch_tiles(echo_graph g, int32_t max_tiles) {
    g_last_error.clear();
    if (!g) return fail(ECHO_ERR_ARG, "null graph");
    if (max_tiles < 0) return fail(ECHO_ERR_ARG, "max_tiles %d < 0", max_tiles);
    g->max_launch_tiles = max_tiles;
    return ECHO_OK;
}

int echo_walk_chain(echo_graph g, const int64_t weight_ps[3], int64_t out[4]) {
    g_last_error.clear();
    if (!g || !weight_ps || !out) return fail(ECHO_ERR_ARG, "null argument");
    for (int i = 0; i < 3; ++i)
        if (weight_ps[i] < 0 || weight_ps[i] >= (int64_t(1) << 40))
            return fail(ECHO_ERR_ARG, "weight %d = %lld outside [0, 2^40)", i, (long long)weight_ps[i]);
    try {
        return walk_chain(g, weight_ps, out);
    } catch (const std::bad_alloc &) {
        return fail(ECHO_ERR_NOMEM, "host allocation failed while following the walk lists");
    }
}

const char *echo_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
