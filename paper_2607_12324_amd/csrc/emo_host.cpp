// Host side of the EMO policy-evaluation library: argument checking, graph analysis (merging
// duplicate edges, Kahn topological sort with depths, cycle detection), folding of nodes whose
// finish time does not depend on the candidate, compilation of the graph into kernel programs,
// device upload, and the C ABI entry points declared in include/emo.h.
//
// The canonical topological order reported by emo_graph_topo_order sorts nodes by (depth, id)
// (the traversal order of Alg. 1).  The kernels may walk any topological order: the forward
// recurrence (Eq. 1) takes exact maxima and one rounded addition per node, so every
// topological order yields bit-identical finish times.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <limits>
#include <memory>
#include <mutex>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "emo.h"
#include "emo_internal.h"

namespace {

thread_local std::string g_last_error;

emo_status fail(emo_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

emo_status ok() {
    g_last_error.clear();
    return EMO_OK;
}

}  // namespace

namespace emo {
emo_status report(emo_status s, const char *message) {
    if (s == EMO_OK) {
        g_last_error.clear();
    } else {
        g_last_error = message;
    }
    return s;
}
}  // namespace emo

namespace {

emo_status device_fail(hipError_t e, const char *where) {
    return fail(EMO_ERR_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

// Topological schedule of a traversal: the node of each step and, per step, the steps of its
// candidate-dependent predecessors and successors.
struct Schedule {
    std::vector<int32_t> seq;
    std::vector<std::vector<int32_t>> in, out;
    std::vector<float> cst;      // latest finish among candidate-independent predecessors
    bool monotone = true;        // packs in increasing id
};

// Interpreter program compiled on the host before upload.
struct HostProgram {
    std::vector<emo::FwdStep> fwd;
    std::vector<uint32_t> ins;
    std::vector<emo::BwdStep> bwd;
    std::vector<uint32_t> succs;
    int32_t n_cold = 0, n_cold_bwd = 0, n_hot = 0, n_hot_bwd = 0;
    float t_const = 0.f;
    bool monotone = true;
};

// A value read again within this many steps is kept in the register bank when a slot is free.
constexpr int32_t kHotSpan = 96;

constexpr int32_t kJitMaxOps = 2048;      // larger graphs compile too slowly as one kernel
constexpr int32_t kJitMaxSlackOps = 160;  // every finish time stays in a VGPR
// Segmented kernels (larger graphs): steps per segment kernel and per recompute sub-segment,
// and the largest graph compiled this way (compile time grows with the step count).
constexpr int32_t kChainSegOps = 256;
constexpr int32_t kChainSubOps = 32;
constexpr int32_t kChainMaxOps = 8192;
// Slack on disjoint stream chains in the windowed layout takes the chain scan, not the segmented
// kernels, from this many steps on: measured on 16 chains, the scan takes 0.51 ms against 0.66
// for 1,024 packs and 262,144 candidates, 1.51 against 1.75 for 768 packs and 2^20 candidates,
// but 1.17 against 1.11 for 512 packs.
constexpr int32_t kChainScanMinOps = 768;
// Cut-segment kernels: packs per segment at most, packs per recompute sub-segment.
constexpr int32_t kCutMaxPacks = 256;
constexpr int32_t kCutSubPacks = 32;
// ... and only for graphs of small cut width: the finish times live at once in the forward pass
// are held in registers (wider graphs keep the interpreting kernels, which spill cold values to
// device scratch by design).
constexpr int32_t kChainMaxLive = 48;
constexpr size_t kJitTableLds = 64 * 1024;
constexpr size_t kJitTableLdsSlack = 40 * 1024;

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    bool active = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
            if (hipSetDevice(dev) == hipSuccess) active = true;
        }
    }
    ~DeviceGuard() {
        if (active) (void)hipSetDevice(prev);
    }
};

// Device scratch reused across batch calls (selection partials, checkpoint rows, cold slots):
// allocated on first need, grown (never shrunk) on demand, freed with its owner.  Each of the
// first kStreamSlots streams that call gets a buffer of its own: calls on one stream are
// ordered by the stream, so they reuse it with no event and no host wait (an event record per
// call cost about 4 us of device time between kernels), and growing waits for that stream,
// which is live since it is the caller's.  Calls from further streams share one buffer: a call
// on another stream than the previous one first waits for the event recorded after that
// call's kernels, and growing waits for it on the host before the old buffer is freed.
// Steady-state calls allocate and free nothing, so the host keeps launching ahead of the
// device.
constexpr int kStreamSlots = 8;

struct Arena {
    struct Slot {
        hipStream_t s = nullptr;
        void *ptr = nullptr;
        size_t bytes = 0;
    };
    std::mutex mu;
    Slot slots[kStreamSlots];
    int nslots = 0;
    // the shared buffer of calls from further streams
    void *ptr = nullptr;
    size_t bytes = 0;
    hipEvent_t done = nullptr;   // recorded after the last shared call's kernels
    hipStream_t last = nullptr;
    bool used = false;
    bool shared_call = false;    // the current call uses the shared buffer
};

size_t grown(size_t need, size_t have) { return std::max(need, have + have / 4); }

// With a.mu held and the arena's device current: at least `bytes` of scratch for a call on s.
hipError_t arena_acquire(Arena &a, size_t bytes, hipStream_t s, void **out) {
    hipError_t e = hipSuccess;
    a.shared_call = false;
    for (int i = 0; i < a.nslots; ++i) {
        Arena::Slot &sl = a.slots[i];
        if (sl.s != s) continue;
        if (bytes > sl.bytes) {
            if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;   // earlier calls on s
            const size_t want = grown(bytes, sl.bytes);
            (void)hipFree(sl.ptr);
            sl.ptr = nullptr;
            sl.bytes = 0;
            if ((e = hipMalloc(&sl.ptr, want)) != hipSuccess) {
                sl.ptr = nullptr;
                return e;
            }
            sl.bytes = want;
        }
        *out = sl.ptr;
        return hipSuccess;
    }
    if (a.nslots < kStreamSlots) {
        Arena::Slot &sl = a.slots[a.nslots];
        if ((e = hipMalloc(&sl.ptr, bytes)) != hipSuccess) {
            sl.ptr = nullptr;
            return e;
        }
        sl.s = s;
        sl.bytes = bytes;
        ++a.nslots;
        *out = sl.ptr;
        return hipSuccess;
    }
    a.shared_call = true;
    if (!a.done && (e = hipEventCreateWithFlags(&a.done, hipEventDisableTiming)) != hipSuccess) return e;
    if (bytes > a.bytes) {
        if (a.used && (e = hipEventSynchronize(a.done)) != hipSuccess) return e;
        const size_t want = grown(bytes, a.bytes);
        if (a.ptr) (void)hipFree(a.ptr);
        a.ptr = nullptr;
        a.bytes = 0;
        if ((e = hipMalloc(&a.ptr, want)) != hipSuccess) {
            a.ptr = nullptr;
            return e;
        }
        a.bytes = want;
    } else if (a.used && a.last != s) {
        if ((e = hipStreamWaitEvent(s, a.done, 0)) != hipSuccess) return e;
    }
    *out = a.ptr;
    return hipSuccess;
}

// With a.mu held: marks the end of the call's kernels on s (shared buffer only).
hipError_t arena_release(Arena &a, hipStream_t s) {
    if (!a.shared_call) return hipSuccess;
    a.used = true;
    a.last = s;
    return hipEventRecord(a.done, s);
}

void arena_free(Arena &a) {
    for (int i = 0; i < a.nslots; ++i)
        if (a.slots[i].ptr) (void)hipFree(a.slots[i].ptr);
    a.nslots = 0;
    if (a.done) (void)hipEventDestroy(a.done);
    if (a.ptr) (void)hipFree(a.ptr);
    a.done = nullptr;
    a.ptr = nullptr;
    a.bytes = 0;
    a.used = false;
}

}  // namespace

struct emo_graph_s {
    int32_t V = 0, E = 0, P = 0, F = 1;
    float static_power = 0.f;
    int32_t device = -1;
    std::vector<int32_t> src, dst;           // merged edges
    std::vector<int32_t> pack;
    std::vector<float> dur;
    std::vector<int32_t> pred_off, pred, succ_off, succ;
    std::vector<int32_t> order, depth;       // canonical order, depths
    std::vector<int32_t> kahn;               // a topological order (Kahn, FIFO)
    std::vector<char> dyn;                   // depends on the candidate
    std::vector<float> const_eft;            // finish time of candidate-independent nodes
    std::vector<float> tmin;                 // each pack's least time over its levels
    float t_const = 0.f;
    emo_graph_info info{};
    std::vector<void *> allocations;         // device memory owned by the handle
    emo::DevGraph dg;
    // graph-specialised kernels
    int32_t kernel_mode = EMO_KERNELS_AUTO;
    emo::JitGraph jg;
    bool jit_eligible = false;
    bool jit_slack_eligible = false;
    bool jit_slack_staged = false;
    std::mutex jit_mu;
    int jit_state = 0;                       // 0 not tried, 1 compiled, -1 failed
    emo::JitModule jm;
    std::string jit_log;
    // segmented kernels: forward kernels for eval/select when one kernel would not hold the
    // table in LDS, backward kernels for slack when the graph is too large to keep every finish
    // time
    bool chain_eval = false;
    bool chain_slack = false;
    bool chain_scan_first = false;           // slack: windowed chain scan before segmented kernels
    int chain_state = 0;                     // 0 not tried, 1 compiled, -1 failed
    emo::JitModule jc;
    emo::DevChains chains;                   // chain-lane program (lanes == 0: not chains)
    // cut-segment kernels
    emo::CutPlan cut_plan;
    bool cut_ok = false;
    int cut_state = 0;                       // 0 not tried, 1 compiled, -1 failed
    emo::JitModule jk;
    // time-interval kernels specialised to the graph
    int iv_state = 0;                        // 0 not tried, 1 compiled, -1 failed
    emo::JitModule jiv;
    int64_t iv_cap_key = -1, iv_cap = 0;     // resident workgroups for the last (K, M)
    Arena arena;                             // per-call scratch, kept between calls
    Arena dp_arena;                          // scratch of the policy search (whose evaluations
                                             // use `arena`)
    // profiling hook (hipEvent_t handles owned by the caller)
    hipEvent_t ev_begin = nullptr;
    hipEvent_t ev_end = nullptr;
};

namespace {

// CSR adjacency: for each node, the list of `from` endpoints of edges ending there.
void build_csr(int32_t V, const std::vector<int32_t> &from, const std::vector<int32_t> &to,
               std::vector<int32_t> &off, std::vector<int32_t> &adj) {
    off.assign(static_cast<size_t>(V) + 1, 0);
    for (int32_t t : to) off[t + 1]++;
    for (int32_t v = 0; v < V; ++v) off[v + 1] += off[v];
    adj.assign(from.size(), 0);
    std::vector<int32_t> fill(off.begin(), off.end() - 1);
    for (size_t i = 0; i < from.size(); ++i) adj[fill[to[i]]++] = from[i];
}

// Kahn's algorithm (FIFO): a topological order and depths (longest path in edges).
emo_status topo_sort(emo_graph_s &g) {
    const int32_t V = g.V;
    std::vector<int32_t> indeg(V, 0);
    for (int32_t v = 0; v < V; ++v) indeg[v] = g.pred_off[v + 1] - g.pred_off[v];
    g.kahn.clear();
    g.kahn.reserve(V);
    g.depth.assign(V, 0);
    for (int32_t v = 0; v < V; ++v)
        if (indeg[v] == 0) g.kahn.push_back(v);
    for (size_t head = 0; head < g.kahn.size(); ++head) {
        int32_t v = g.kahn[head];
        for (int32_t j = g.succ_off[v]; j < g.succ_off[v + 1]; ++j) {
            int32_t u = g.succ[j];
            g.depth[u] = std::max(g.depth[u], g.depth[v] + 1);
            if (--indeg[u] == 0) g.kahn.push_back(u);
        }
    }
    if (static_cast<int32_t>(g.kahn.size()) != V)
        return fail(EMO_ERR_CYCLE, "the graph has a cycle (%d of %d nodes are orderable)",
                    static_cast<int>(g.kahn.size()), static_cast<int>(V));
    // canonical order: stable bucket sort of node ids by depth
    int32_t maxd = 0;
    for (int32_t v = 0; v < V; ++v) maxd = std::max(maxd, g.depth[v]);
    std::vector<int32_t> cnt(static_cast<size_t>(maxd) + 2, 0);
    for (int32_t v = 0; v < V; ++v) cnt[g.depth[v] + 1]++;
    for (int32_t d = 0; d <= maxd; ++d) cnt[d + 1] += cnt[d];
    g.order.assign(V, 0);
    for (int32_t v = 0; v < V; ++v) g.order[cnt[g.depth[v]]++] = v;
    g.info.max_depth = V ? maxd : 0;
    return EMO_OK;
}

// Drops edges implied by longer paths: u -> v goes when another path leads from u to v (found
// by a search over the merged graph that only visits nodes placed before the last other
// predecessor of v, within a visit budget; an edge not proven implied stays).  Durations are
// >= 0 and rounding is monotone, so finish times do not decrease along a path and latest start
// times do not increase against it, also in fp32: such an edge never decides the maximum of
// Eq. 1 nor the minimum of the backward pass, and every EFT, LFT and slack is unchanged, bit
// for bit.  Fewer edges mean fewer operations and shorter live ranges in the kernels.  The
// removable edges are decided on the merged graph, so reachability is preserved (the result
// lies between the graph and its transitive reduction).  Returns the number of dropped edges.
int32_t prune_implied_edges(emo_graph_s &g) {
    const int32_t V = g.V;
    std::vector<int32_t> pos(V);
    for (int32_t i = 0; i < V; ++i) pos[g.order[i]] = i;
    std::vector<int32_t> stamp(V, -1), target(V, -1), stack;
    std::vector<char> drop(g.src.size(), 0);
    // merged edge behind predecessor slot j (build_csr fills the slots in edge order)
    std::vector<int32_t> edge_of(g.pred.size());
    {
        std::vector<int32_t> fill(g.pred_off.begin(), g.pred_off.end() - 1);
        for (size_t e = 0; e < g.src.size(); ++e) edge_of[fill[g.dst[e]]++] = static_cast<int32_t>(e);
    }
    int64_t budget = 64 * (static_cast<int64_t>(V) + static_cast<int64_t>(g.src.size())) + 65536;
    constexpr int32_t kQueryVisits = 4096;
    int32_t query = 0, dropped = 0;
    std::vector<int32_t> preds;
    for (int32_t v = 0; v < V && budget > 0; ++v) {
        const int32_t b = g.pred_off[v], e = g.pred_off[v + 1];
        if (e - b < 2) continue;
        int32_t top = -1, second = -1;   // the two largest predecessor positions
        for (int32_t j = b; j < e; ++j) {
            const int32_t p = pos[g.pred[j]];
            target[g.pred[j]] = v;
            if (p > top) { second = top; top = p; }
            else if (p > second) second = p;
        }
        for (int32_t j = b; j < e && budget > 0; ++j) {
            const int32_t u = g.pred[j];
            const int32_t lim = pos[u] == top ? second : top;
            if (lim <= pos[u]) continue;   // no other predecessor comes after u
            ++query;
            bool found = false;
            int32_t visits = 0;
            stack.assign(1, u);
            stamp[u] = query;
            while (!stack.empty() && !found && visits < kQueryVisits) {
                const int32_t x = stack.back();
                stack.pop_back();
                ++visits;
                for (int32_t k = g.succ_off[x]; k < g.succ_off[x + 1]; ++k) {
                    const int32_t y = g.succ[k];
                    if (pos[y] > lim || stamp[y] == query) continue;
                    // y is another predecessor of v: u reaches v by a path of two or more edges
                    if (target[y] == v) { found = true; break; }
                    stamp[y] = query;
                    stack.push_back(y);
                }
            }
            budget -= visits;
            if (found) {
                drop[edge_of[j]] = 1;
                ++dropped;
            }
        }
    }
    if (dropped == 0) return 0;
    std::vector<int32_t> src, dst;
    for (size_t i = 0; i < g.src.size(); ++i)
        if (!drop[i]) {
            src.push_back(g.src[i]);
            dst.push_back(g.dst[i]);
        }
    build_csr(V, src, dst, g.pred_off, g.pred);
    build_csr(V, dst, src, g.succ_off, g.succ);
    return dropped;
}

// Marks candidate-dependent nodes and computes the fp32 finish times of the others.
void fold_constants(emo_graph_s &g) {
    const int32_t V = g.V;
    g.dyn.assign(V, 0);
    g.const_eft.assign(V, 0.f);
    float tc = 0.f;
    for (int32_t v : g.kahn) {
        bool d = g.pack[v] >= 0;
        float est = 0.f;
        for (int32_t j = g.pred_off[v]; j < g.pred_off[v + 1]; ++j) {
            int32_t k = g.pred[j];
            if (g.dyn[k]) d = true;
            else est = std::max(est, g.const_eft[k]);
        }
        g.dyn[v] = d;
        if (!d) {
            g.const_eft[v] = est + g.dur[v];
            tc = std::max(tc, g.const_eft[v]);
        }
    }
    g.t_const = tc;
}


// Topological order of the traversal.  fold: only candidate-dependent nodes become steps.
// Ready nodes are taken by (key, id) with key = pack id for packs and -1 for fixed nodes, so
// packs are visited in increasing pack id whenever the pack numbering is consistent with the
// precedence edges.
Schedule make_schedule(const emo_graph_s &g, bool fold) {
    Schedule sc;
    const int32_t V = g.V;
    auto included = [&](int32_t v) { return !fold || g.dyn[v]; };
    std::vector<int32_t> indeg(V, 0);
    for (int32_t v = 0; v < V; ++v) {
        if (!included(v)) continue;
        for (int32_t j = g.pred_off[v]; j < g.pred_off[v + 1]; ++j)
            if (included(g.pred[j])) indeg[v]++;
    }
    using Key = std::pair<int64_t, int32_t>;
    std::priority_queue<Key, std::vector<Key>, std::greater<Key>> ready;
    auto key = [&](int32_t v) -> int64_t { return g.pack[v] >= 0 ? g.pack[v] : -1; };
    for (int32_t v = 0; v < V; ++v)
        if (included(v) && indeg[v] == 0) ready.push({key(v), v});
    while (!ready.empty()) {
        int32_t v = ready.top().second;
        ready.pop();
        sc.seq.push_back(v);
        for (int32_t j = g.succ_off[v]; j < g.succ_off[v + 1]; ++j) {
            int32_t u = g.succ[j];
            if (included(u) && --indeg[u] == 0) ready.push({key(u), u});
        }
    }
    const int32_t n = static_cast<int32_t>(sc.seq.size());
    std::vector<int32_t> pos(V, -1);
    for (int32_t i = 0; i < n; ++i) pos[sc.seq[i]] = i;
    sc.in.resize(n);
    sc.out.resize(n);
    sc.cst.assign(n, 0.f);
    int32_t last_pack = -1;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t v = sc.seq[i];
        for (int32_t j = g.pred_off[v]; j < g.pred_off[v + 1]; ++j) {
            const int32_t k = g.pred[j];
            if (included(k)) sc.in[i].push_back(pos[k]);
            else sc.cst[i] = std::max(sc.cst[i], g.const_eft[k]);
        }
        for (int32_t j = g.succ_off[v]; j < g.succ_off[v + 1]; ++j)
            if (included(g.succ[j])) sc.out[i].push_back(pos[g.succ[j]]);
        if (g.pack[v] >= 0) {
            if (g.pack[v] < last_pack) sc.monotone = false;
            last_pack = g.pack[v];
        }
    }
    return sc;
}

// Hot (register bank) and cold (device scratch) slot pools; the lowest free index is reused.
struct SlotPool {
    std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> hot_free, cold_free;
    int32_t next_hot = 0, next_cold = 0;
    uint32_t acquire(bool want_hot) {
        if (want_hot) {
            if (!hot_free.empty()) {
                int32_t h = hot_free.top();
                hot_free.pop();
                return static_cast<uint32_t>(h);
            }
            if (next_hot < emo::kHotSlots) return static_cast<uint32_t>(next_hot++);
        }
        int32_t c;
        if (!cold_free.empty()) {
            c = cold_free.top();
            cold_free.pop();
        } else {
            c = next_cold++;
        }
        return emo::kColdRef | static_cast<uint32_t>(c);
    }
    void release(uint32_t ref) {
        if (ref & emo::kColdRef) cold_free.push(static_cast<int32_t>(ref & ~emo::kColdRef));
        else hot_free.push(static_cast<int32_t>(ref));
    }
};

uint32_t fbits(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return u;
}

// Interpreter program for a schedule.  backward: add the reverse pass (slack); per_node: slack
// columns are node ids, else pack ids.
HostProgram compile_program(const emo_graph_s &g, const Schedule &sc, bool fold, bool backward,
                            bool per_node) {
    HostProgram hp;
    const int32_t n = static_cast<int32_t>(sc.seq.size());
    hp.t_const = fold ? g.t_const : 0.f;
    hp.monotone = sc.monotone;
    // forward: a finish time stays live until its last reader
    std::vector<int32_t> last_use(n, -1);
    for (int32_t i = 0; i < n; ++i)
        for (int32_t k : sc.in[i]) last_use[k] = std::max(last_use[k], i);
    std::vector<uint32_t> ref(n, 0);
    SlotPool pool;
    hp.fwd.resize(n);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t v = sc.seq[i];
        emo::FwdStep st{};
        st.pack = g.pack[v];
        st.cst = fbits(sc.cst[i]);
        st.dur = fbits(g.pack[v] >= 0 ? 0.f : g.dur[v]);
        st.in_begin = static_cast<int32_t>(hp.ins.size());
        st.in_count = static_cast<int32_t>(sc.in[i].size());
        for (int32_t k : sc.in[i]) hp.ins.push_back(ref[k]);
        for (int32_t k : sc.in[i])
            if (last_use[k] == i) pool.release(ref[k]);
        if (sc.out[i].empty()) st.flags |= emo::kStepSink;
        if (last_use[i] >= 0) {
            ref[i] = pool.acquire(last_use[i] - i <= kHotSpan);
            st.flags |= emo::kStepOut;
            st.out = ref[i];
        }
        hp.fwd[i] = st;
    }
    hp.n_cold = pool.next_cold;
    hp.n_hot = pool.next_hot;
    if (!backward) return hp;
    // backward: a latest start time stays live until its first predecessor (in forward order)
    std::vector<int32_t> first_pred(n, -1);
    for (int32_t i = 0; i < n; ++i)
        if (!sc.in[i].empty()) first_pred[i] = *std::min_element(sc.in[i].begin(), sc.in[i].end());
    std::vector<uint32_t> bref(n, 0);
    SlotPool bpool;
    hp.bwd.reserve(n);
    for (int32_t i = n - 1; i >= 0; --i) {
        const int32_t v = sc.seq[i];
        emo::BwdStep st{};
        st.pack = g.pack[v];
        st.dur = fbits(g.pack[v] >= 0 ? 0.f : g.dur[v]);
        st.succ_begin = static_cast<int32_t>(hp.succs.size());
        st.succ_count = static_cast<int32_t>(sc.out[i].size());
        for (int32_t u : sc.out[i]) hp.succs.push_back(bref[u]);
        for (int32_t u : sc.out[i])
            if (first_pred[u] == i) bpool.release(bref[u]);
        if (first_pred[i] >= 0) {
            bref[i] = bpool.acquire(i - first_pred[i] <= kHotSpan);
            st.flags |= emo::kStepOut;
            st.out = bref[i];
        }
        st.col = per_node ? v : g.pack[v];
        st.fwd = i;
        hp.bwd.push_back(st);
    }
    hp.n_cold_bwd = bpool.next_cold;
    hp.n_hot_bwd = bpool.next_hot;
    return hp;
}

template <typename T>
emo_status upload(emo_graph_s &g, const std::vector<T> &host, const T **dev) {
    size_t bytes = std::max<size_t>(host.size() * sizeof(T), 16);
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) return fail(EMO_ERR_OUT_OF_MEMORY, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
    g.allocations.push_back(p);
    if (!host.empty()) {
        e = hipMemcpy(p, host.data(), host.size() * sizeof(T), hipMemcpyHostToDevice);
        if (e != hipSuccess) return device_fail(e, "hipMemcpy");
    }
    *dev = static_cast<const T *>(p);
    return EMO_OK;
}

emo_status upload_program(emo_graph_s &g, const HostProgram &hp, emo::DevProgram &dp) {
    dp.n_ops = static_cast<int32_t>(hp.fwd.size());
    dp.n_cold = hp.n_cold;
    dp.n_cold_bwd = hp.n_cold_bwd;
    dp.t_const = hp.t_const;
    dp.monotone = hp.monotone ? 1 : 0;
    emo_status s;
    if ((s = upload(g, hp.fwd, &dp.fwd)) != EMO_OK) return s;
    if ((s = upload(g, hp.ins, &dp.ins)) != EMO_OK) return s;
    if ((s = upload(g, hp.bwd, &dp.bwd)) != EMO_OK) return s;
    if ((s = upload(g, hp.succs, &dp.succs)) != EMO_OK) return s;
    return EMO_OK;
}

void release_device(emo_graph_s *g) {
    if (g->device >= 0) {
        DeviceGuard guard(g->device);
        emo::jit_unload(&g->jm);
        emo::jit_unload(&g->jc);
        emo::jit_unload(&g->jk);
        for (void *p : g->allocations) (void)hipFree(p);
        arena_free(g->arena);
        arena_free(g->dp_arena);
    }
    g->allocations.clear();
}

bool is_pow2(int32_t x) { return x > 0 && (x & (x - 1)) == 0; }

// Chain-lane program of a folded schedule whose steps form disjoint chains (at most one
// candidate-dependent predecessor and successor each) and at most 64 of them: steps[k][lane]
// is the k-th step of chain `lane`, padded with steps that leave a finish time unchanged.
// Returns false when the schedule does not have that shape.
// Windowed layout of the chains (see DevChains): steps grouped by the window of their pack (a
// fixed node stays in the window of the chain's previous pack, window 0 before the first), one
// block per window.  Takes the widest window (256, 128, ... 16 packs) whose working set fits.
// Returns false when some chain goes back to an earlier window or no window width fits.
bool build_chain_windows(const emo_graph_s &g, const Schedule &sc,
                         const std::vector<std::vector<int32_t>> &chains,
                         std::vector<uint4> *blocks, emo::DevChains *dc) {
    const int32_t nc = static_cast<int32_t>(chains.size());
    // (level offsets within a workgroup's rows are 32-bit: at most 1024 rows of P bytes; rows of
    // a pack count that is not a multiple of 16 are copied from the dwords around each piece)
    if (nc < 1 || nc > 16 || g.P < 16 || g.P >= (1 << 21)) return false;
    const int32_t hdr_words = (nc + 1 + 3) / 4 * 4;
    for (int32_t W = 256; W >= 16; W >>= 1) {
        const int32_t nwin = (g.P + W - 1) / W;
        // window of every step
        std::vector<std::vector<int32_t>> win(nc);
        bool monotone = true;
        int32_t fixed = 0;
        for (int32_t c = 0; c < nc && monotone; ++c) {
            int32_t w = 0;
            for (int32_t i : chains[c]) {
                const int32_t p = g.pack[sc.seq[i]];
                if (p >= 0) {
                    if (p / W < w) {
                        monotone = false;
                        break;
                    }
                    w = p / W;
                } else {
                    fixed = 1;
                }
                win[c].push_back(w);
            }
        }
        if (!monotone) return false;   // narrower windows would not be monotone either
        // records per window: 8 no-op steps on each side (reads run up to two groups of 4 past
        // a chain's range) and each chain's steps padded to a multiple of 4
        std::vector<int32_t> per(static_cast<size_t>(nwin) * nc, 0);
        for (int32_t c = 0; c < nc; ++c)
            for (int32_t w : win[c]) ++per[static_cast<size_t>(w) * nc + c];
        int32_t rec_max = 0;
        for (int32_t w = 0; w < nwin; ++w) {
            int32_t n = 16;
            for (int32_t c = 0; c < nc; ++c) n += (per[static_cast<size_t>(w) * nc + c] + 3) / 4 * 4;
            rec_max = std::max(rec_max, n);
        }
        const int32_t blk_bytes = 4 * hdr_words + 16 * rec_max;
        int32_t G = 0;
        if (!emo::chain_window_fits(nc, g.F, W, blk_bytes, g.P % 16 == 0, &G)) continue;
        const size_t words = static_cast<size_t>(blk_bytes) / 4;
        emo::ChainWinStep noop;
        noop.ct = static_cast<uint32_t>(W) | (static_cast<uint32_t>(W * g.F) << 16);
        noop.cst = 0.f;
        noop.dur = 0.f;
        noop.pad = 0u;
        std::vector<uint32_t> buf(static_cast<size_t>(nwin) * words, 0u);
        for (int32_t w = 0; w < nwin; ++w)
            for (int32_t r = 0; r < rec_max; ++r)
                std::memcpy(&buf[static_cast<size_t>(w) * words + hdr_words + 4 * static_cast<size_t>(r)], &noop,
                            sizeof(noop));
        // chain after chain: chain c's records of window w follow those of chains < c
        std::vector<int32_t> fill(nwin, 8);   // next record per window
        for (int32_t c = 0; c < nc; ++c) {
            for (int32_t w = 0; w < nwin; ++w) buf[static_cast<size_t>(w) * words + c] = static_cast<uint32_t>(fill[w]);
            for (size_t k = 0; k < chains[c].size(); ++k) {
                const int32_t i = chains[c][k];
                const int32_t v = sc.seq[i];
                const int32_t p = g.pack[v];
                const int32_t w = win[c][k];
                const uint32_t col = static_cast<uint32_t>(p >= 0 ? p - w * W : W);
                emo::ChainWinStep st;
                st.ct = col | ((col * static_cast<uint32_t>(g.F)) << 16);
                st.cst = sc.cst[i];
                st.dur = p >= 0 ? 0.f : g.dur[v];
                st.pad = 0u;
                std::memcpy(&buf[static_cast<size_t>(w) * words + hdr_words + 4 * static_cast<size_t>(fill[w])],
                            &st, sizeof(st));
                ++fill[w];
            }
            for (int32_t w = 0; w < nwin; ++w) fill[w] = (fill[w] + 3) / 4 * 4;
        }
        for (int32_t w = 0; w < nwin; ++w) buf[static_cast<size_t>(w) * words + nc] = static_cast<uint32_t>(fill[w]);
        blocks->assign(buf.size() / 4, make_uint4(0u, 0u, 0u, 0u));
        std::memcpy(blocks->data(), buf.data(), buf.size() * sizeof(uint32_t));
        dc->nc = nc;
        dc->win = W;
        dc->nwin = nwin;
        dc->groups = G;
        dc->fixed = fixed;
        dc->hdr_words = hdr_words;
        dc->blk_bytes = blk_bytes;
        // per-thread plans of chains_scan_full: NC = 64 G candidates, 64 G nc threads and
        // NC * W / 4 float4 pieces of the slack tile per window
        // (and the copy slots that kernel is compiled for: one level piece, one or two forward
        // and one second-pass table pieces and one step-block piece per thread)
        const int64_t NC = 64 * static_cast<int64_t>(G);
        const int64_t nthr = 64 * static_cast<int64_t>(G) * nc;
        const int64_t tab8 = (static_cast<int64_t>(W) * g.F / 2 + nthr - 1) / nthr;
        const int64_t tab4 = (static_cast<int64_t>(W) * g.F / 4 + nthr - 1) / nthr;
        const bool slots = NC * (W / 16) <= nthr && (tab8 == 1 || tab8 == 2) && tab4 == 1 && blk_bytes / 16 <= nthr;
        dc->full = slots && g.P % W == 0 && NC * W / 4 <= 4 * nthr &&
                           NC * g.P * 4 < (int64_t(1) << 31) &&
                           static_cast<int64_t>(g.P) * g.F * 8 < (int64_t(1) << 31) &&
                           static_cast<int64_t>(nwin) * blk_bytes < (int64_t(1) << 31)
                       ? 1
                       : 0;
        return true;
    }
    return false;
}

bool build_chains(const emo_graph_s &g, const Schedule &sc, std::vector<emo::ChainStep> *steps,
                  std::vector<int32_t> *pos, emo::DevChains *dc, std::vector<uint4> *blocks) {
    const int32_t n = static_cast<int32_t>(sc.seq.size());
    if (n == 0) return false;
    std::vector<int32_t> heads;
    for (int32_t i = 0; i < n; ++i) {
        if (sc.in[i].size() > 1 || sc.out[i].size() > 1) return false;
        if (sc.in[i].empty()) heads.push_back(i);
    }
    const int32_t C = static_cast<int32_t>(heads.size());
    if (C < 1 || C > 64) return false;
    std::vector<std::vector<int32_t>> chains(C);
    size_t longest = 0;
    for (int32_t c = 0; c < C; ++c) {
        for (int32_t i = heads[c];; i = sc.out[i][0]) {
            chains[c].push_back(i);
            if (sc.out[i].empty()) break;
        }
        longest = std::max(longest, chains[c].size());
    }
    int32_t lanes = 1, lane_log = 0;
    while (lanes < C) {
        lanes <<= 1;
        ++lane_log;
    }
    const int32_t len = static_cast<int32_t>((longest + emo::kChainStepBlock - 1) / emo::kChainStepBlock *
                                             emo::kChainStepBlock);
    steps->assign(static_cast<size_t>(len) * lanes, emo::ChainStep{-1, 0.f, 0.f, 0});
    pos->assign(static_cast<size_t>(g.P), 0);
    for (int32_t c = 0; c < C; ++c)
        for (size_t k = 0; k < chains[c].size(); ++k) {
            const int32_t i = chains[c][k];
            const int32_t v = sc.seq[i];
            emo::ChainStep &st = (*steps)[k * lanes + c];
            st.pack = g.pack[v];
            st.cst = sc.cst[i];
            st.dur = g.pack[v] >= 0 ? 0.f : g.dur[v];
            if (g.pack[v] >= 0) (*pos)[g.pack[v]] = static_cast<int32_t>(k * lanes + c);
        }
    dc->lanes = lanes;
    dc->lane_log = lane_log;
    dc->len = len;
    dc->t_const = g.t_const;
    if (!build_chain_windows(g, sc, chains, blocks, dc)) {
        dc->win = 0;
        blocks->clear();
    }
    return true;
}

// The specialised kernels' view of the graph: the folded schedule's steps, with predecessors
// and successors as step indices.
emo::JitGraph make_jit_graph(const emo_graph_s &g, const Schedule &sc) {
    emo::JitGraph jg;
    jg.P = g.P;
    jg.F = g.F;
    jg.static_power = g.static_power;
    jg.t_const = g.t_const;
    jg.pack_monotone = sc.monotone;
    const size_t n = sc.seq.size();
    jg.ops.resize(n);
    for (size_t i = 0; i < n; ++i) {
        emo::JitOp &o = jg.ops[i];
        const int32_t v = sc.seq[i];
        o.pack = g.pack[v];
        o.cst = sc.cst[i];
        o.dur = g.pack[v] >= 0 ? 0.f : g.dur[v];
        o.in = sc.in[i];
        o.out = sc.out[i];
    }
    return jg;
}

// Steps that are cut nodes: nodes that every other node precedes or follows.  At position i of
// a topological order that holds exactly when no edge jumps over position i, no node before it
// is a sink and no node after it is a source.  Returns their step indices in increasing order.
std::vector<int32_t> cut_steps(const emo_graph_s &g, const Schedule &sf) {
    const int32_t V = g.V;
    std::vector<int32_t> pos(V), jump(static_cast<size_t>(V) + 1, 0), step(V, -1);
    for (int32_t i = 0; i < V; ++i) pos[g.order[i]] = i;
    for (int32_t u = 0; u < V; ++u)
        for (int32_t k = g.succ_off[u]; k < g.succ_off[u + 1]; ++k) {
            const int32_t a = pos[u], b = pos[g.succ[k]];
            if (b > a + 1) {
                jump[a + 1]++;
                jump[b]--;
            }
        }
    for (size_t i = 0; i < sf.seq.size(); ++i) step[sf.seq[i]] = static_cast<int32_t>(i);
    std::vector<char> source_after(static_cast<size_t>(V) + 1, 0);
    for (int32_t i = V - 1; i >= 0; --i) {
        const int32_t v = g.order[i];
        source_after[i] = source_after[i + 1] || g.pred_off[v] == g.pred_off[v + 1];
    }
    std::vector<int32_t> cuts;
    bool sink_before = false;
    int32_t over = 0;
    for (int32_t i = 0; i < V; ++i) {
        over += jump[i];
        const int32_t v = g.order[i];
        if (over == 0 && !sink_before && !source_after[i + 1] && step[v] >= 0) cuts.push_back(step[v]);
        sink_before = sink_before || g.succ_off[v] == g.succ_off[v + 1];
    }
    std::sort(cuts.begin(), cuts.end());
    return cuts;
}

// Whether every sum and difference of durations along paths is an exact fp32 number, whatever
// the order of the additions: all time values (table times and fixed durations) are multiples
// of one power of two u, and the longest path with every pack at its largest duration is below
// 2^24 u.  Every finish time, start floor, partial sum along a path and makespan of any policy
// is then a multiple of u below 2^24 u (durations only lengthen paths), and so is the
// difference of two of them.
bool exact_time_sums(const emo_graph_s &g, const float *pack_time) {
    int emin = INT_MAX;
    auto visit = [&](float x) {
        if (x <= 0.f) return;
        int e = 0;
        const float m = std::frexp(x, &e);
        const uint32_t M = static_cast<uint32_t>(std::ldexp(m, 24));
        emin = std::min(emin, e - 24 + __builtin_ctz(M));
    };
    std::vector<double> longest(static_cast<size_t>(g.V), 0.0);
    double T = 0.0;
    for (int32_t i = 0; i < g.V; ++i) {
        const int32_t v = g.order[i];
        double d = 0.0;
        if (g.pack[v] >= 0) {
            for (int32_t f = 0; f < g.F; ++f) {
                const float x = pack_time[static_cast<size_t>(g.pack[v]) * g.F + f];
                visit(x);
                d = std::max(d, static_cast<double>(x));
            }
        } else {
            visit(g.dur[v]);
            d = g.dur[v];
        }
        double start = 0.0;
        for (int32_t j = g.pred_off[v]; j < g.pred_off[v + 1]; ++j) start = std::max(start, longest[g.pred[j]]);
        longest[v] = start + d;
        T = std::max(T, longest[v]);
    }
    return emin == INT_MAX || T < std::ldexp(1.0, 24 + emin);
}

size_t jit_table_bytes(const emo_graph_s &g) {
    return (static_cast<size_t>(g.P) * g.F + (is_pow2(g.F) ? 0 : emo::kTablePad)) * sizeof(float2);
}

// Source of the specialised kernels and the workgroup size they are written for.
std::string jit_source(const emo_graph_s &g, int *block_out) {
    const size_t tb = jit_table_bytes(g);
    const bool with_slack = g.jit_slack_eligible;
    const bool tab_lds = tb <= (with_slack ? kJitTableLdsSlack : kJitTableLds);
    // one LDS copy of a large table serves a larger workgroup
    const int block = !tab_lds || tb <= 16 * 1024 ? 256 : (tb <= 32 * 1024 ? 512 : 1024);
    *block_out = block;
    return emo::jit_generate(g.jg, with_slack, tab_lds, block);
}

// Generates and compiles the time-interval kernels once; returns 1 when they are ready.
int ensure_iv(emo_graph_s *g) {
    std::lock_guard<std::mutex> lock(g->jit_mu);
    if (g->iv_state != 0) return g->iv_state;
    const size_t tb = static_cast<size_t>(g->P) * g->F * sizeof(float2);
    const bool tab_lds = tb <= kJitTableLds;
    const std::string src = emo::jit_generate_intervals(g->jg, tab_lds, 256);
    DeviceGuard guard(g->device);
    emo::JitModule m;
    std::string log;
    if (emo::jit_compile_intervals(src, &m, &log) != 0) {
        g->jit_log = log;
        g->iv_state = -1;
        return -1;
    }
    m.block = 256;
    g->jiv = m;
    g->iv_state = 1;
    g->info.compile_seconds += static_cast<float>(m.compile_seconds);
    return 1;
}

// Bucket table parameters of the time-interval kernels for change points p_0 < ... < p_{K-2}: a
// scale with distinct floor(fl(p_j * scale)) (the exact fp32 product the kernel forms) and
// M = the largest such bucket + 2.  False when that needs more than kIvMaxBuckets buckets.
bool iv_buckets(const float *pts, int K, float *scale_out, int *M_out) {
    if (K <= 1) {
        *scale_out = 0.f;
        *M_out = 1;
        return true;
    }
    double gap = INFINITY;
    for (int i = 0; i + 2 < K; ++i) gap = std::min(gap, static_cast<double>(pts[i + 1]) - pts[i]);
    if (K == 2) gap = pts[0];
    for (double c : {1.01, 1.25, 2.0, 4.0}) {
        const float s = static_cast<float>(c / gap);
        if (!(s > 0.f) || !std::isfinite(s)) continue;
        const float top = pts[K - 2] * s;
        if (!(top < static_cast<float>(emo::kIvMaxBuckets - 2))) continue;
        bool distinct = true;
        for (int i = 0; i + 2 < K && distinct; ++i)
            distinct = static_cast<int>(pts[i] * s) < static_cast<int>(pts[i + 1] * s);
        if (!distinct) continue;
        *scale_out = s;
        *M_out = static_cast<int>(top) + 2;
        return true;
    }
    return false;
}

// Generates and compiles the specialised kernels once; returns 1 when they are ready.
int ensure_jit(emo_graph_s *g) {
    std::lock_guard<std::mutex> lock(g->jit_mu);
    if (g->jit_state != 0) return g->jit_state;
    int block = 256;
    std::string src = jit_source(*g, &block);
    DeviceGuard guard(g->device);
    emo::JitModule m;
    std::string log;
    if (emo::jit_compile(src, g->jit_slack_eligible, &m, &log) != 0) {
        g->jit_log = log;
        g->jit_state = -1;
        g->info.specialized |= 4;
        return -1;
    }
    m.block = block;
    // persistent workgroups pay off when each one copies a large table into LDS
    if (jit_table_bytes(*g) > 16 * 1024) emo::jit_set_caps(&m);
    g->jm = m;
    g->jit_state = 1;
    g->info.specialized |= 1 | (m.slack ? 2 : 0);
    g->info.compile_seconds += static_cast<float>(m.compile_seconds);
    return 1;
}

emo::ChainPlan chain_plan(const emo_graph_s &g) {
    return emo::jit_chain_plan(g.jg, g.chain_slack, kChainSegOps, kChainSubOps);
}

// Generates and compiles the segmented kernels once; returns 1 when they are ready.
int ensure_chain(emo_graph_s *g) {
    std::lock_guard<std::mutex> lock(g->jit_mu);
    if (g->chain_state != 0) return g->chain_state;
    const emo::ChainPlan cp = chain_plan(*g);
    const std::string src = emo::jit_generate_chain(g->jg, cp);
    DeviceGuard guard(g->device);
    emo::JitModule m;
    std::string log;
    if (emo::jit_compile_chain(src, cp, &m, &log) != 0) {
        g->jit_log = log;
        g->chain_state = -1;
        g->info.specialized |= 4;
        return -1;
    }
    g->jc = m;
    g->chain_state = 1;
    g->info.specialized |= 8 | (g->chain_eval ? 1 : 0) | (g->chain_slack ? 2 : 0);
    g->info.compile_seconds += static_cast<float>(m.compile_seconds);
    return 1;
}

// Generates and compiles the cut-segment kernels once; returns 1 when they are ready.
int ensure_cut(emo_graph_s *g) {
    std::lock_guard<std::mutex> lock(g->jit_mu);
    if (g->cut_state != 0) return g->cut_state;
    const std::string src = emo::jit_generate_cut(g->jg, g->cut_plan);
    DeviceGuard guard(g->device);
    emo::JitModule m;
    std::string log;
    if (emo::jit_compile_cut(src, g->cut_plan, &m, &log) != 0) {
        g->jit_log = log;
        g->cut_state = -1;
        g->info.specialized |= 4;
        return -1;
    }
    g->jk = m;
    g->cut_state = 1;
    g->info.specialized |= 16;
    g->info.compile_seconds += static_cast<float>(m.compile_seconds);
    return 1;
}

bool aligned(const void *p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }

// Which kernels a batch call uses (the value of emo_graph_info.last_kernels, except that the
// windowed form of the chain lanes reports 4).
enum class Path { kInterpreted = 0, kSingle = 1, kChain = 2, kChainLanes = 3, kCut = 5 };

// Chooses the kernels of a batch call, compiling specialised kernels on first use.  Returns
// EMO_OK and sets *path, or an error in EMO_KERNELS_SPECIALIZED mode.
emo_status choose_path(emo_graph_s *g, const uint8_t *levels, const float *slack, bool per_node,
                       int64_t B, Path *path) {
    *path = Path::kInterpreted;
    if (g->kernel_mode == EMO_KERNELS_INTERPRETED) return EMO_OK;
    if (slack && per_node) return EMO_OK;   // per-node slack: interpreted kernels only
    if (slack && g->chain_scan_first && !g->jit_slack_eligible &&
        emo::chains_windowed_ok(g->chains, levels, slack)) {
        *path = Path::kChainLanes;
        return EMO_OK;
    }
    // disjoint chains too long for the segmented kernels: one lane per chain
    const bool chain_lanes = g->chains.lanes > 0 && !(slack ? g->jit_slack_eligible || g->chain_slack
                                                            : g->jit_eligible || g->chain_eval);
    if (chain_lanes) {
        *path = Path::kChainLanes;
        return EMO_OK;
    }
    // graphs with cut nodes, too large for one kernel (or, without slack, for its table in LDS):
    // the segments between cuts in parallel (ahead of the segmented kernels: 1,024 packs with 4
    // cuts, 2^20 candidates without slack, take 0.28 ms there against 0.35)
    const bool single_ok = slack ? g->jit_slack_eligible : g->jit_eligible && !g->chain_eval;
    if (!single_ok && g->cut_ok && B < (int64_t(1) << 30) && aligned(levels, 16) &&
        (!slack || aligned(slack, 16))) {
        if (ensure_cut(g) == 1) {
            *path = Path::kCut;
            return EMO_OK;
        }
        if (g->kernel_mode == EMO_KERNELS_SPECIALIZED)
            return fail(EMO_ERR_DEVICE, "cut-segment kernels failed to compile: %.400s", g->jit_log.c_str());
    }
    if (!aligned(levels, static_cast<size_t>(emo::jit_level_width(g->jg)))) return EMO_OK;
    bool single = false, chain = false;
    if (slack) {
        single = g->jit_slack_eligible;
        chain = !single && g->chain_slack;
    } else {
        chain = g->chain_eval;
        single = !chain && g->jit_eligible;
    }
    if (!single && !chain) return EMO_OK;
    const int st = single ? ensure_jit(g) : ensure_chain(g);
    if (st != 1) {
        if (g->kernel_mode == EMO_KERNELS_SPECIALIZED)
            return fail(EMO_ERR_DEVICE, "specialised kernels failed to compile: %.400s", g->jit_log.c_str());
        return EMO_OK;
    }
    if (single && slack && (!g->jm.slack || (g->jit_slack_staged && !aligned(slack, 16)))) return EMO_OK;
    if (chain && slack && g->jc.plan.staged && !aligned(slack, 16)) return EMO_OK;
    *path = single ? Path::kSingle : Path::kChain;
    return EMO_OK;
}

bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.f; }

emo_status check_batch(emo_graph_t g, int64_t B) {
    if (!g) return fail(EMO_ERR_INVALID_ARGUMENT, "graph handle is NULL");
    if (g->device < 0) return fail(EMO_ERR_UNSUPPORTED, "graph was loaded host-only (device -1)");
    if (B < 0 || B >= (int64_t(1) << 32))
        return fail(EMO_ERR_INVALID_ARGUMENT, "num_candidates %lld outside [0, 2^32)", (long long)B);
    return EMO_OK;
}

emo_status after_launch(hipError_t e, const char *what) {
    if (e != hipSuccess) return device_fail(e, what);
    return ok();
}

}  // namespace

extern "C" {

const char *emo_status_string(emo_status s) {
    switch (s) {
        case EMO_OK: return "EMO_OK";
        case EMO_ERR_INVALID_ARGUMENT: return "EMO_ERR_INVALID_ARGUMENT";
        case EMO_ERR_CYCLE: return "EMO_ERR_CYCLE";
        case EMO_ERR_OUT_OF_MEMORY: return "EMO_ERR_OUT_OF_MEMORY";
        case EMO_ERR_DEVICE: return "EMO_ERR_DEVICE";
        case EMO_ERR_UNSUPPORTED: return "EMO_ERR_UNSUPPORTED";
    }
    return "EMO_ERR_UNKNOWN";
}

const char *emo_last_error(void) { return g_last_error.c_str(); }

emo_status emo_load_graph(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                          const int32_t *edge_dst, const int32_t *node_pack,
                          const float *node_duration, int32_t num_packs, int32_t num_levels,
                          const float *pack_time, const float *pack_energy, float static_power,
                          int32_t device, emo_graph_t *out) {
    if (!out) return fail(EMO_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    const int32_t V = num_nodes, E = num_edges, P = num_packs, F = num_levels;
    if (V < 0 || E < 0 || P < 0) return fail(EMO_ERR_INVALID_ARGUMENT, "negative size");
    if (F < 1 || F > 256) return fail(EMO_ERR_INVALID_ARGUMENT, "num_levels %d outside [1, 256]", F);
    if (P > V) return fail(EMO_ERR_INVALID_ARGUMENT, "more packs (%d) than nodes (%d)", P, V);
    if (E > 0 && (!edge_src || !edge_dst)) return fail(EMO_ERR_INVALID_ARGUMENT, "edge arrays are NULL");
    if (V > 0 && (!node_pack || !node_duration)) return fail(EMO_ERR_INVALID_ARGUMENT, "node arrays are NULL");
    if (P > 0 && (!pack_time || !pack_energy)) return fail(EMO_ERR_INVALID_ARGUMENT, "table arrays are NULL");
    if (int64_t(P) * F > (int64_t(1) << 28)) return fail(EMO_ERR_INVALID_ARGUMENT, "tables too large");
    if (!finite_nonneg(static_power)) return fail(EMO_ERR_INVALID_ARGUMENT, "static_power must be finite and >= 0");
    if (device < -1) return fail(EMO_ERR_INVALID_ARGUMENT, "device %d", device);
    if (device >= 0) {
        int n = 0;
        hipError_t e = hipGetDeviceCount(&n);
        if (e != hipSuccess || device >= n)
            return fail(EMO_ERR_DEVICE, "device %d not available (%d devices)", device, n);
    }
    for (int32_t i = 0; i < E; ++i) {
        if (edge_src[i] < 0 || edge_src[i] >= V || edge_dst[i] < 0 || edge_dst[i] >= V)
            return fail(EMO_ERR_INVALID_ARGUMENT, "edge %d (%d -> %d) out of range", i, edge_src[i], edge_dst[i]);
        if (edge_src[i] == edge_dst[i]) return fail(EMO_ERR_CYCLE, "self-loop on node %d", edge_src[i]);
    }
    std::vector<int32_t> seen(P, 0);
    for (int32_t v = 0; v < V; ++v) {
        int32_t p = node_pack[v];
        if (p < -1 || p >= P) return fail(EMO_ERR_INVALID_ARGUMENT, "node %d has pack id %d outside [-1, %d)", v, p, P);
        if (p >= 0) {
            if (seen[p]++) return fail(EMO_ERR_INVALID_ARGUMENT, "pack %d appears on more than one node", p);
        } else if (!finite_nonneg(node_duration[v])) {
            return fail(EMO_ERR_INVALID_ARGUMENT, "node %d duration must be finite and >= 0", v);
        }
    }
    for (int32_t p = 0; p < P; ++p)
        if (!seen[p]) return fail(EMO_ERR_INVALID_ARGUMENT, "pack %d is on no node", p);
    for (int64_t i = 0; i < int64_t(P) * F; ++i)
        if (!finite_nonneg(pack_time[i]) || !finite_nonneg(pack_energy[i]))
            return fail(EMO_ERR_INVALID_ARGUMENT, "table entry %lld must be finite and >= 0", (long long)i);

    emo_graph_s *g = new (std::nothrow) emo_graph_s();
    if (!g) return fail(EMO_ERR_OUT_OF_MEMORY, "host allocation");
    std::unique_ptr<emo_graph_s, void (*)(emo_graph_s *)> holder(g, [](emo_graph_s *x) {
        release_device(x);
        delete x;
    });
    g->V = V; g->P = P; g->F = F; g->static_power = static_power; g->device = device;
    g->pack.assign(node_pack, node_pack + V);
    g->dur.assign(node_duration, node_duration + V);
    g->tmin.assign(P, 0.f);
    for (int32_t p = 0; p < P; ++p) {
        float m = pack_time[static_cast<size_t>(p) * F];
        for (int32_t f = 1; f < F; ++f) m = std::min(m, pack_time[static_cast<size_t>(p) * F + f]);
        g->tmin[p] = m;
    }
    for (int32_t v = 0; v < V; ++v)
        if (g->pack[v] >= 0) g->dur[v] = 0.f;
    // merge duplicate edges
    {
        std::vector<int64_t> keys(E);
        for (int32_t i = 0; i < E; ++i) keys[i] = int64_t(edge_src[i]) * V + edge_dst[i];
        std::sort(keys.begin(), keys.end());
        keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
        g->src.resize(keys.size());
        g->dst.resize(keys.size());
        for (size_t i = 0; i < keys.size(); ++i) {
            g->src[i] = static_cast<int32_t>(keys[i] / V);
            g->dst[i] = static_cast<int32_t>(keys[i] % V);
        }
        g->E = static_cast<int32_t>(keys.size());
    }
    build_csr(V, g->src, g->dst, g->pred_off, g->pred);
    build_csr(V, g->dst, g->src, g->succ_off, g->succ);
    emo_status s = topo_sort(*g);
    if (s != EMO_OK) return s;
    const int32_t implied = prune_implied_edges(*g);
    fold_constants(*g);

    const Schedule sf = make_schedule(*g, true);
    const Schedule sa = make_schedule(*g, false);
    HostProgram pe = compile_program(*g, sf, true, false, false);
    HostProgram ps = compile_program(*g, sf, true, true, false);
    HostProgram pn = compile_program(*g, sa, false, true, true);

    emo_graph_info &in = g->info;
    in.num_nodes = V; in.num_edges = g->E; in.num_packs = P; in.num_levels = F;
    in.num_implied_edges = implied;
    in.num_dynamic_nodes = static_cast<int32_t>(pe.fwd.size());
    in.num_dynamic_edges = static_cast<int32_t>(pe.ins.size());
    in.eval_slots = pe.n_hot + pe.n_cold;
    in.const_makespan = g->t_const;
    in.device = device;
    in.pack_order_monotone = sf.monotone ? 1 : 0;
    in.kernel_mode = EMO_KERNELS_AUTO;
    g->jg = make_jit_graph(*g, sf);
    std::vector<emo::ChainStep> csteps;
    std::vector<int32_t> cpos;
    std::vector<uint4> cblocks;
    emo::DevChains dc;
    const bool exact_sums = exact_time_sums(*g, pack_time);
    const bool chains_ok = build_chains(*g, sf, &csteps, &cpos, &dc, &cblocks);
    in.chain_lanes = chains_ok ? dc.lanes : 0;
    in.chain_window = chains_ok ? dc.win : 0;
    in.chain_scan_window = chains_ok ? dc.win : 0;
    in.chain_scan_full = chains_ok && dc.win > 0 && dc.full ? 1 : 0;
    const int32_t nops = static_cast<int32_t>(sf.seq.size());
    g->jit_eligible = nops >= 1 && nops <= kJitMaxOps;
    g->jit_slack_eligible = g->jit_eligible && nops <= kJitMaxSlackOps;
    g->jit_slack_staged = sf.monotone && P % 16 == 0;
    const bool narrow = pe.n_hot + pe.n_cold <= kChainMaxLive;
    // Without slack, one kernel past kJitTableLds reads the table from global memory: the
    // segmented kernels (table windows in LDS) are then faster whenever the live set allows.  At
    // 2^20 candidates and 16 levels, 640 steps on 16 chains (an 80 KB table) take 0.26 ms there
    // against 0.93 ms in one kernel, 2,048 steps 0.82 against 3.84; 512 steps (64 KB, in LDS)
    // take 0.14 ms in one kernel against 0.19.
    g->chain_eval = narrow && nops <= kChainMaxOps && (nops > kJitMaxOps || jit_table_bytes(*g) > kJitTableLds);
    g->chain_slack = narrow && nops > kJitMaxSlackOps && nops <= kChainMaxOps;
    g->chain_scan_first = chains_ok && dc.win > 0 && nops >= kChainScanMinOps;
    g->cut_plan = emo::jit_cut_plan(g->jg, cut_steps(*g, sf), kCutMaxPacks, kCutSubPacks);
    // (off the exact-sum grid the segment-local times round differently from the program order
    // of the other kinds: results agree with them to rounding, not bit for bit)
    g->cut_ok = g->cut_plan.segments() >= 2 && nops <= kChainMaxOps;
    in.cut_segments = g->cut_ok ? g->cut_plan.segments() : 0;
    in.exact_time_sums = exact_sums ? 1 : 0;
    int rt = 0;
    in.hip_runtime_version = hipRuntimeGetVersion(&rt) == hipSuccess ? rt : 0;

    if (device >= 0) {
        DeviceGuard guard(device);
        std::vector<float2> tab(static_cast<size_t>(P) * F + emo::kTablePad, make_float2(0.f, 0.f));
        for (size_t i = 0; i < static_cast<size_t>(P) * F; ++i)
            tab[i] = make_float2(pack_time[i], pack_energy[i]);
        g->dg.V = V; g->dg.P = P; g->dg.F = F; g->dg.static_power = static_power;
        if ((s = upload(*g, tab, &g->dg.tab)) != EMO_OK) return s;
        std::vector<float> tabt(tab.size());
        for (size_t i = 0; i < tab.size(); ++i) tabt[i] = tab[i].x;
        if ((s = upload(*g, tabt, &g->dg.tabt)) != EMO_OK) return s;
        if ((s = upload_program(*g, pe, g->dg.eval)) != EMO_OK) return s;
        if ((s = upload_program(*g, ps, g->dg.slack_pack)) != EMO_OK) return s;
        if ((s = upload_program(*g, pn, g->dg.slack_node)) != EMO_OK) return s;
        if (chains_ok) {
            if ((s = upload(*g, csteps, &dc.steps)) != EMO_OK) return s;
            if ((s = upload(*g, cpos, &dc.pos)) != EMO_OK) return s;
            if (dc.win > 0 && (s = upload(*g, cblocks, &dc.blocks)) != EMO_OK) return s;
            g->chains = dc;
        }
    }
    *out = holder.release();
    return ok();
}

emo_status emo_free_graph(emo_graph_t g) {
    if (!g) return ok();
    release_device(g);
    delete g;
    return ok();
}

emo_status emo_graph_get_info(emo_graph_t g, emo_graph_info *info) {
    if (!g || !info) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    *info = g->info;
    return ok();
}

emo_status emo_graph_set_kernel_mode(emo_graph_t g, int32_t mode) {
    if (!g) return fail(EMO_ERR_INVALID_ARGUMENT, "graph handle is NULL");
    if (mode != EMO_KERNELS_AUTO && mode != EMO_KERNELS_INTERPRETED && mode != EMO_KERNELS_SPECIALIZED)
        return fail(EMO_ERR_INVALID_ARGUMENT, "unknown kernel mode %d", mode);
    g->kernel_mode = mode;
    g->info.kernel_mode = mode;
    return ok();
}

emo_status emo_graph_set_timing_events(emo_graph_t g, void *begin_event, void *end_event) {
    if (!g) return fail(EMO_ERR_INVALID_ARGUMENT, "graph handle is NULL");
    g->ev_begin = static_cast<hipEvent_t>(begin_event);
    g->ev_end = static_cast<hipEvent_t>(end_event);
    return ok();
}

emo_status emo_graph_specialized_source(emo_graph_t g, char *buf, int64_t *len) {
    if (!g || !len) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    if (!g->jit_eligible) return fail(EMO_ERR_UNSUPPORTED, "graph too large for one specialised kernel");
    int block = 256;
    std::string src = jit_source(*g, &block);
    const int64_t need = static_cast<int64_t>(src.size()) + 1;
    if (!buf) {
        *len = need;
        return ok();
    }
    if (*len < need) return fail(EMO_ERR_INVALID_ARGUMENT, "buffer of %lld bytes, %lld needed",
                                 (long long)*len, (long long)need);
    std::memcpy(buf, src.c_str(), static_cast<size_t>(need));
    *len = need;
    return ok();
}

emo_status emo_graph_segmented_source(emo_graph_t g, char *buf, int64_t *len) {
    if (!g || !len) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    if (!g->chain_eval && !g->chain_slack)
        return fail(EMO_ERR_UNSUPPORTED, "the graph uses no segmented kernels");
    const std::string src = emo::jit_generate_chain(g->jg, chain_plan(*g));
    const int64_t need = static_cast<int64_t>(src.size()) + 1;
    if (!buf) {
        *len = need;
        return ok();
    }
    if (*len < need) return fail(EMO_ERR_INVALID_ARGUMENT, "buffer of %lld bytes, %lld needed",
                                 (long long)*len, (long long)need);
    std::memcpy(buf, src.c_str(), static_cast<size_t>(need));
    *len = need;
    return ok();
}

emo_status emo_graph_cut_source(emo_graph_t g, char *buf, int64_t *len) {
    if (!g || !len) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    if (!g->cut_ok) return fail(EMO_ERR_UNSUPPORTED, "the graph has no cut segments");
    const std::string src = emo::jit_generate_cut(g->jg, g->cut_plan);
    const int64_t need = static_cast<int64_t>(src.size()) + 1;
    if (!buf) {
        *len = need;
        return ok();
    }
    if (*len < need) return fail(EMO_ERR_INVALID_ARGUMENT, "buffer of %lld bytes, %lld needed",
                                 (long long)*len, (long long)need);
    std::memcpy(buf, src.c_str(), static_cast<size_t>(need));
    *len = need;
    return ok();
}

emo_status emo_graph_interval_source(emo_graph_t g, char *buf, int64_t *len) {
    if (!g || !len) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    if (!g->jit_eligible) return fail(EMO_ERR_UNSUPPORTED, "graph too large for one specialised kernel");
    const size_t tb = static_cast<size_t>(g->P) * g->F * sizeof(float2);
    const std::string src = emo::jit_generate_intervals(g->jg, tb <= kJitTableLds, 256);
    const int64_t need = static_cast<int64_t>(src.size()) + 1;
    if (!buf) {
        *len = need;
        return ok();
    }
    if (*len < need) return fail(EMO_ERR_INVALID_ARGUMENT, "buffer of %lld bytes, %lld needed",
                                 (long long)*len, (long long)need);
    std::memcpy(buf, src.c_str(), static_cast<size_t>(need));
    *len = need;
    return ok();
}

emo_status emo_graph_topo_order(emo_graph_t g, int32_t *order, int32_t *depth) {
    if (!g || (!order && g->V > 0)) return fail(EMO_ERR_INVALID_ARGUMENT, "NULL argument");
    if (g->V > 0) std::memcpy(order, g->order.data(), sizeof(int32_t) * g->V);
    if (depth && g->V > 0) std::memcpy(depth, g->depth.data(), sizeof(int32_t) * g->V);
    return ok();
}

}  // extern "C"

namespace {

constexpr int kMaxDevices = 64;

// Scratch of calls that have no graph handle, one arena per device.
Arena &device_arena(int dev) {
    static Arena arenas[kMaxDevices];
    return arenas[dev];
}

// Checks nt latency targets with their optional masks and results (nt == 0: none) and fills
// tg's targets and masks; tg.n stays 0 when no target has a mask or a result.
emo_status check_targets(int32_t nt, const float *targets, uint32_t *const *masks,
                         emo_selection *results, emo::SelTargets *tg) {
    if (nt < 0 || nt > emo::kMaxTargets)
        return fail(EMO_ERR_INVALID_ARGUMENT, "num_targets %d outside [0, %d]", nt, emo::kMaxTargets);
    if (results && reinterpret_cast<uintptr_t>(results) % 8)
        return fail(EMO_ERR_INVALID_ARGUMENT, "result is not 8-byte aligned");
    bool any = results != nullptr;
    for (int32_t k = 0; k < nt && masks; ++k) any = any || masks[k];
    if (!any || nt == 0) return ok();
    if (!targets) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_targets is NULL");
    for (int32_t k = 0; k < nt; ++k) {
        if (std::isnan(targets[k])) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_target %d is NaN", k);
        tg->t[k] = targets[k];
        tg->mask[k] = masks ? masks[k] : nullptr;
    }
    tg->n = nt;
    return ok();
}

// The hot path for every batch entry point: forward pass, optional backward slack pass, and for
// each of nt latency targets an optional feasibility mask and selection, in one evaluating
// kernel launch (the selection's stage 1 inside it) plus one finalize launch for all targets.
emo_status evaluate(emo_graph_t g, const uint8_t *levels, int64_t B, float *makespan,
                    float *energy, float *slack, int32_t per_node, int32_t nt, const float *targets,
                    uint32_t *const *masks, emo_selection *results, void *stream) {
    emo_status s = check_batch(g, B);
    if (s != EMO_OK) return s;
    emo::SelTargets tg;
    if ((s = check_targets(nt, targets, masks, results, &tg)) != EMO_OK) return s;
    if (!tg.n) results = nullptr;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (B == 0) {
        if (!results) return ok();
        DeviceGuard guard(g->device);
        hipError_t e = hipSuccess;
        for (int32_t k = 0; k < tg.n && e == hipSuccess; ++k) e = emo::launch_empty_result(results + k, st);
        return after_launch(e, "empty selection");
    }
    if (!makespan && !energy && !slack && !tg.n) return ok();
    if (!levels && g->P > 0) return fail(EMO_ERR_INVALID_ARGUMENT, "levels is NULL");
    Path path = Path::kInterpreted;
    if ((s = choose_path(g, levels, slack, per_node != 0, B, &path)) != EMO_OK) return s;
    DeviceGuard guard(g->device);
    // one selection partial record per block of the evaluating kernel
    const int64_t nblocks = path == Path::kSingle  ? emo::jit_blocks(g->jm, B)
                            : path == Path::kChain ? emo::jit_chain_blocks(g->jc, B)
                            : path == Path::kCut   ? emo::jit_cut_blocks(g->jk, B)
                            : path == Path::kChainLanes ? emo::select_results_blocks(B)
                                                   : emo::forward_blocks(B);
    const emo::DevProgram &prog = per_node ? g->dg.slack_node : g->dg.slack_pack;
    size_t part_bytes = results ? static_cast<size_t>(tg.n) * nblocks * emo::kPartialBytes : 0;
    part_bytes = (part_bytes + 255) & ~static_cast<size_t>(255);
    size_t work_bytes = 0;
    if (path == Path::kChain) work_bytes = emo::chain_scratch_bytes(g->jc.plan, B);
    else if (path == Path::kCut) work_bytes = emo::cut_scratch_bytes(g->jk.cut_plan, B);
    else if (path == Path::kChainLanes) work_bytes = emo::chains_scratch_bytes(g->dg, g->chains, levels, B, slack);
    else if (path == Path::kInterpreted)
        work_bytes = slack ? emo::slack_scratch_bytes(prog, B) : emo::forward_scratch_bytes(g->dg.eval, B);
    std::lock_guard<std::mutex> lock(g->arena.mu);
    void *scratch = nullptr;
    if (part_bytes + work_bytes > 0) {
        hipError_t ea = arena_acquire(g->arena, part_bytes + work_bytes, st, &scratch);
        if (ea != hipSuccess) {
            (void)hipGetLastError();
            return fail(EMO_ERR_OUT_OF_MEMORY, "scratch of %zu bytes: %s", part_bytes + work_bytes,
                        hipGetErrorString(ea));
        }
    }
    tg.part = results ? scratch : nullptr;
    tg.nparts = nblocks;
    void *work = scratch ? static_cast<char *>(scratch) + part_bytes : nullptr;
    g->info.last_kernels = path == Path::kChainLanes && emo::chains_scan_full_ok(g->chains, levels, slack)
                               ? 8
                               : path == Path::kChainLanes && emo::chains_scan_ok(g->chains, levels, slack)
                               ? 6
                               : path == Path::kChainLanes && emo::chains_windowed_ok(g->chains, levels, slack)
                                     ? 4
                                     : static_cast<int32_t>(path);
    hipError_t e = g->ev_begin ? hipEventRecord(g->ev_begin, st) : hipSuccess;
    if (e == hipSuccess) {
        if (path == Path::kCut) {
            e = emo::jit_launch_cut(g->jk, levels, B, g->dg.tab, work, slack, makespan, energy, tg, st);
        } else if (path == Path::kChain) {
            e = emo::jit_launch_chain(g->jc, levels, B, g->dg.tab, g->dg.tabt, work, slack, makespan,
                                      energy, tg, st);
        } else if (path == Path::kChainLanes) {
            e = emo::launch_chains(g->dg, g->chains, levels, B, makespan, energy, slack, tg, work, st);
        } else if (slack) {
            if (path == Path::kSingle) {
                e = emo::jit_launch_slack(g->jm, levels, B, g->dg.tab, slack, makespan, energy, tg, st);
            } else {
                e = emo::launch_slack(g->dg, prog, per_node ? g->V : g->P, levels, B, slack,
                                      makespan, energy, tg, work, st);
            }
        } else if (path == Path::kSingle) {
            e = emo::jit_launch_forward(g->jm, levels, B, g->dg.tab, makespan, energy, tg, st);
        } else {
            e = emo::launch_forward(g->dg, levels, B, makespan, energy, tg, work, st);
        }
    }
    if (e == hipSuccess && g->ev_end) e = hipEventRecord(g->ev_end, st);
    if (results && e == hipSuccess) e = emo::launch_select_finalize(tg, results, st);
    if (scratch) {
        hipError_t er = arena_release(g->arena, st);
        if (e == hipSuccess) e = er;
    }
    return after_launch(e, "evaluation");
}

}  // namespace

extern "C" {

emo_status emo_eval_policies(emo_graph_t g, const uint8_t *levels, int64_t B, float *makespan,
                             float *energy, void *stream) {
    return evaluate(g, levels, B, makespan, energy, nullptr, 0, 0, nullptr, nullptr, nullptr, stream);
}

emo_status emo_slack(emo_graph_t g, const uint8_t *levels, int64_t B, float *slack,
                     int32_t per_node, float *makespan, float *energy, void *stream) {
    if (!slack && B > 0) return fail(EMO_ERR_INVALID_ARGUMENT, "slack is NULL");
    return evaluate(g, levels, B, makespan, energy, slack, per_node, 0, nullptr, nullptr, nullptr, stream);
}

emo_status emo_select_policy(emo_graph_t g, const uint8_t *levels, int64_t B,
                             float latency_target, uint32_t *feasible_mask,
                             emo_selection *result, void *stream) {
    if (!result) return fail(EMO_ERR_INVALID_ARGUMENT, "result is NULL");
    return evaluate(g, levels, B, nullptr, nullptr, nullptr, 0, 1, &latency_target, &feasible_mask,
                    result, stream);
}

emo_status emo_evaluate(emo_graph_t g, const uint8_t *levels, int64_t B, float *makespan,
                        float *energy, float *slack, int32_t per_node, float latency_target,
                        uint32_t *feasible_mask, emo_selection *result, void *stream) {
    return evaluate(g, levels, B, makespan, energy, slack, per_node, 1, &latency_target,
                    &feasible_mask, result, stream);
}

emo_status emo_evaluate_targets(emo_graph_t g, const uint8_t *levels, int64_t B, float *makespan,
                                float *energy, float *slack, int32_t per_node, int32_t num_targets,
                                const float *latency_targets, uint32_t *const *feasible_masks,
                                emo_selection *results, void *stream) {
    if (num_targets < 1 || num_targets > emo::kMaxTargets)
        return fail(EMO_ERR_INVALID_ARGUMENT, "num_targets %d outside [1, %d]", num_targets, emo::kMaxTargets);
    if (!latency_targets) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_targets is NULL");
    return evaluate(g, levels, B, makespan, energy, slack, per_node, num_targets, latency_targets,
                    feasible_masks, results, stream);
}

emo_status emo_eval_intervals(emo_graph_t g, const uint8_t *levels, int64_t B, int32_t num_intervals,
                              const float *change_points, const float *idle_power, float *makespan,
                              float *energy, float latency_target, uint32_t *feasible_mask,
                              emo_selection *result, void *stream) {
    emo_status s = check_batch(g, B);
    if (s != EMO_OK) return s;
    if (num_intervals < 1 || num_intervals > emo::kMaxIntervals)
        return fail(EMO_ERR_INVALID_ARGUMENT, "num_intervals %d outside [1, %d]", num_intervals,
                    emo::kMaxIntervals);
    if (num_intervals > 1 && !change_points) return fail(EMO_ERR_INVALID_ARGUMENT, "change_points is NULL");
    if (!idle_power) return fail(EMO_ERR_INVALID_ARGUMENT, "idle_power is NULL");
    emo::IvPolicy pol;
    pol.K = num_intervals;
    for (int i = 0; i + 1 < num_intervals; ++i) {
        const float t = change_points[i];
        if (!std::isfinite(t) || t <= 0.f || (i > 0 && !(t > change_points[i - 1])))
            return fail(EMO_ERR_INVALID_ARGUMENT,
                        "change point %d (%g) is not finite, positive and above the previous one", i, (double)t);
        pol.pts[i] = t;
    }
    for (int f = 0; f < emo::kMaxLevels; ++f) pol.idle[f] = 0.f;
    for (int f = 0; f < g->F; ++f) {
        if (!finite_nonneg(idle_power[f]))
            return fail(EMO_ERR_INVALID_ARGUMENT, "idle_power[%d] is negative or not finite", f);
        pol.idle[f] = idle_power[f];
    }
    emo::SelTargets tg;
    if ((s = check_targets(1, &latency_target, &feasible_mask, result, &tg)) != EMO_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    DeviceGuard guard(g->device);
    if (B == 0) return result ? after_launch(emo::launch_empty_result(result, st), "empty selection") : ok();
    if (!makespan && !energy && !tg.n) return ok();
    if (!levels) return fail(EMO_ERR_INVALID_ARGUMENT, "levels is NULL");
    // straight-line kernels specialised to the graph when it is small enough for one kernel and
    // the change points fit the bucket table; otherwise the interpreting kernel
    emo::IvJitArgs iva;
    bool use_jit = g->kernel_mode != EMO_KERNELS_INTERPRETED && g->jit_eligible &&
                   iv_buckets(pol.pts, num_intervals, &iva.scale, &iva.M);
    if (use_jit) {
        const int st = ensure_iv(g);
        if (st != 1 && g->kernel_mode == EMO_KERNELS_SPECIALIZED)
            return fail(EMO_ERR_DEVICE, "time-interval kernel compilation failed: %s", g->jit_log.c_str());
        // the rows and the bucket table must fit the workgroup's LDS beside the static tables
        use_jit = st == 1 && g->jiv.iv_static_lds + emo::jit_iv_dyn_lds(g->jiv.block, num_intervals, iva.M) <=
                                 static_cast<size_t>(g->jiv.iv_max_lds);
    }
    int64_t iv_cap = 0;
    if (use_jit) {
        iva.K = num_intervals;
        std::memcpy(iva.pts, pol.pts, sizeof(iva.pts));
        std::memcpy(iva.idle, pol.idle, sizeof(iva.idle));
        // persistent workgroups (each builds the bucket table once): as many as are resident
        const int64_t key = static_cast<int64_t>(num_intervals) << 32 | iva.M;
        std::lock_guard<std::mutex> lock(g->jit_mu);
        if (g->iv_cap_key != key) {
            g->iv_cap = emo::jit_iv_cap(g->jiv, num_intervals, iva.M);
            g->iv_cap_key = key;
        }
        iv_cap = g->iv_cap;
    }
    const int64_t nblocks = use_jit ? emo::jit_blocks(g->jiv, B) : emo::forward_blocks(B);
    size_t part_bytes = result ? static_cast<size_t>(nblocks) * emo::kPartialBytes : 0;
    part_bytes = (part_bytes + 255) & ~static_cast<size_t>(255);
    const size_t work_bytes = use_jit ? 0 : emo::forward_scratch_bytes(g->dg.eval, B);
    std::lock_guard<std::mutex> lock(g->arena.mu);
    void *scratch = nullptr;
    if (part_bytes + work_bytes > 0) {
        hipError_t ea = arena_acquire(g->arena, part_bytes + work_bytes, st, &scratch);
        if (ea != hipSuccess) {
            (void)hipGetLastError();
            return fail(EMO_ERR_OUT_OF_MEMORY, "scratch of %zu bytes: %s", part_bytes + work_bytes,
                        hipGetErrorString(ea));
        }
    }
    tg.part = result ? scratch : nullptr;
    tg.nparts = nblocks;
    void *work = scratch ? static_cast<char *>(scratch) + part_bytes : nullptr;
    g->info.last_kernels = use_jit ? 7 : 0;
    hipError_t e = g->ev_begin ? hipEventRecord(g->ev_begin, st) : hipSuccess;
    if (e == hipSuccess && use_jit)
        e = emo::jit_launch_intervals(g->jiv, levels, B, g->dg.tab, iva, iv_cap, makespan, energy, tg, st);
    else if (e == hipSuccess)
        e = emo::launch_intervals(g->dg, pol, levels, B, makespan, energy, tg, work, st);
    if (e == hipSuccess && g->ev_end) e = hipEventRecord(g->ev_end, st);
    if (result && e == hipSuccess) e = emo::launch_select_finalize(tg, result, st);
    if (scratch) {
        hipError_t er = arena_release(g->arena, st);
        if (e == hipSuccess) e = er;
    }
    return after_launch(e, "emo_eval_intervals");
}

emo_status emo_select_from_results(const float *makespan, const float *energy, int64_t B,
                                   float latency_target, uint32_t *feasible_mask,
                                   emo_selection *result, void *stream) {
    if (B < 0 || B >= (int64_t(1) << 32))
        return fail(EMO_ERR_INVALID_ARGUMENT, "num_candidates %lld outside [0, 2^32)", (long long)B);
    if (!result) return fail(EMO_ERR_INVALID_ARGUMENT, "result is NULL");
    if (reinterpret_cast<uintptr_t>(result) % 8) return fail(EMO_ERR_INVALID_ARGUMENT, "result is not 8-byte aligned");
    if (B > 0 && (!makespan || !energy)) return fail(EMO_ERR_INVALID_ARGUMENT, "makespan/energy is NULL");
    if (std::isnan(latency_target)) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_target is NaN");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (B == 0) return after_launch(emo::launch_empty_result(result, st), "emo_select_from_results");
    const int64_t nblocks = emo::select_results_blocks(B);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(EMO_ERR_DEVICE, "no usable current device (%d)", dev);
    // selection partials live in a per-device arena (kept until the process ends)
    Arena &a = device_arena(dev);
    std::lock_guard<std::mutex> lock(a.mu);
    void *part = nullptr;
    e = arena_acquire(a, static_cast<size_t>(nblocks) * emo::kPartialBytes, st, &part);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(EMO_ERR_OUT_OF_MEMORY, "scratch: %s", hipGetErrorString(e));
    }
    const emo::SelTargets tg = emo::one_target(latency_target, feasible_mask, part, nblocks);
    e = emo::launch_select_results(makespan, energy, B, tg, st);
    if (e == hipSuccess) e = emo::launch_select_finalize(tg, result, st);
    hipError_t er = arena_release(a, st);
    if (e == hipSuccess) e = er;
    return after_launch(e, "emo_select_from_results");
}

emo_status emo_select_from_results_noalloc(const float *makespan, const float *energy,
                                           int64_t B, float latency_target,
                                           uint32_t *feasible_mask, emo_selection *result,
                                           void *stream) {
    if (B < 0 || B > emo::noalloc_max_candidates())
        return fail(EMO_ERR_INVALID_ARGUMENT,
                    "num_candidates %lld outside [0, %lld], the batch the static scratch covers",
                    (long long)B, (long long)emo::noalloc_max_candidates());
    if (!result) return fail(EMO_ERR_INVALID_ARGUMENT, "result is NULL");
    if (reinterpret_cast<uintptr_t>(result) % 8) return fail(EMO_ERR_INVALID_ARGUMENT, "result is not 8-byte aligned");
    if (B > 0 && (!makespan || !energy)) return fail(EMO_ERR_INVALID_ARGUMENT, "makespan/energy is NULL");
    if (std::isnan(latency_target)) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_target is NaN");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (B == 0) return after_launch(emo::launch_empty_result(result, st), "emo_select_from_results_noalloc");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= emo::kNoAllocMaxDevices)
        return fail(EMO_ERR_DEVICE, "no usable current device (%d)", dev);
    void *part = nullptr;
    e = emo::noalloc_scratch(dev, &part);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(EMO_ERR_DEVICE, "static scratch of device %d: %s", dev, hipGetErrorString(e));
    }
    // every partial record is written before the finalize reads it: nothing needs clearing
    const emo::SelTargets tg = emo::one_target(latency_target, feasible_mask, part, emo::select_results_blocks(B));
    e = emo::launch_select_results(makespan, energy, B, tg, st);
    if (e == hipSuccess) e = emo::launch_select_finalize(tg, result, st);
    return after_launch(e, "emo_select_from_results_noalloc");
}

}  // extern "C"

namespace {

// A lower bound of every policy's makespan: the longest path with each pack at its least time
// over the levels (fp64).
double least_makespan(const emo_graph_s &g) {
    std::vector<double> eft(static_cast<size_t>(g.V), 0.0);
    double T = 0.0;
    for (int32_t v : g.order) {
        double est = 0.0;
        for (int32_t j = g.pred_off[v]; j < g.pred_off[v + 1]; ++j) est = std::max(est, eft[g.pred[j]]);
        eft[v] = est + (g.pack[v] >= 0 ? static_cast<double>(g.tmin[g.pack[v]]) : static_cast<double>(g.dur[v]));
        T = std::max(T, eft[v]);
    }
    return T;
}

// Device scratch of one search, carved from one arena block (256-byte aligned pieces): two
// candidate row buffers (this stage's and the next), the stored states after the last stage,
// two key buffers (a stage's source states and its buckets), makespans and energies.
struct DPBuffers {
    uint8_t *rows[2], *state;
    unsigned long long *keys[2];
    float *Tst, *T, *E;
};

size_t dp_layout(int64_t S, int64_t R, int32_t P, DPBuffers *b, char *base) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *p = base ? base + off : nullptr;
        off += (bytes + 255) & ~static_cast<size_t>(255);
        return p;
    };
    const size_t pb = static_cast<size_t>(P > 0 ? P : 1);
    for (int i = 0; i < 2; ++i) {
        b->rows[i] = reinterpret_cast<uint8_t *>(take(static_cast<size_t>(R) * pb));
        b->keys[i] = reinterpret_cast<unsigned long long *>(take(static_cast<size_t>(S) * 8));
    }
    b->state = reinterpret_cast<uint8_t *>(take(static_cast<size_t>(S) * pb));
    b->Tst = reinterpret_cast<float *>(take(static_cast<size_t>(S) * 4));
    b->T = reinterpret_cast<float *>(take(static_cast<size_t>(R) * 4));
    b->E = reinterpret_cast<float *>(take(static_cast<size_t>(R) * 4));
    return off;
}

}  // namespace

extern "C" {

emo_status emo_dp_search(emo_graph_t g, float latency_target, float quantum, const int32_t *pack_order,
                         int32_t max_states, uint8_t *best_levels, emo_selection *result, void *stream) {
    emo_status s = check_batch(g, 1);
    if (s != EMO_OK) return s;
    if (!result || reinterpret_cast<uintptr_t>(result) % 8)
        return fail(EMO_ERR_INVALID_ARGUMENT, "result is NULL or not 8-byte aligned");
    const int32_t P = g->P, F = g->F;
    if (P > 0 && !best_levels) return fail(EMO_ERR_INVALID_ARGUMENT, "best_levels is NULL");
    if (!std::isfinite(latency_target)) return fail(EMO_ERR_INVALID_ARGUMENT, "latency_target must be finite");
    if (!std::isfinite(quantum) || !(quantum > 0.f))
        return fail(EMO_ERR_INVALID_ARGUMENT, "quantum must be finite and > 0");
    if (max_states < 1) return fail(EMO_ERR_INVALID_ARGUMENT, "max_states must be >= 1");
    std::vector<int32_t> order(static_cast<size_t>(P));
    if (pack_order) {
        std::vector<char> seen(static_cast<size_t>(P), 0);
        for (int32_t i = 0; i < P; ++i) {
            const int32_t p = pack_order[i];
            if (p < 0 || p >= P || seen[p]++)
                return fail(EMO_ERR_INVALID_ARGUMENT, "pack_order is not a permutation of the pack ids (entry %d: %d)",
                            i, p);
            order[i] = p;
        }
    } else {
        for (int32_t i = 0; i < P; ++i) order[i] = i;
    }
    // makespan buckets floor(t / q) from one below the least possible makespan's to the target's
    const double q = quantum;
    const int64_t bmin = std::max<int64_t>(0, static_cast<int64_t>(std::floor(least_makespan(*g) / q)) - 1);
    const int64_t btop = static_cast<int64_t>(std::floor(static_cast<double>(latency_target) / q));
    const int64_t NB = std::max<int64_t>(0, btop - bmin + 1);
    if (NB > max_states)
        return fail(EMO_ERR_INVALID_ARGUMENT,
                    "%lld makespan buckets of %g between the least makespan and the target, more than max_states (%d)",
                    (long long)NB, q, max_states);
    const int64_t S = std::max<int64_t>(NB, 1);
    const int64_t R = S * F;
    if (R > (int64_t(1) << 31)) return fail(EMO_ERR_INVALID_ARGUMENT, "too many candidates per stage");
    hipStream_t st = static_cast<hipStream_t>(stream);
    DeviceGuard guard(g->device);
    DPBuffers b{};
    const size_t bytes = dp_layout(S, R, P, &b, nullptr);
    std::lock_guard<std::mutex> lock(g->dp_arena.mu);
    void *base = nullptr;
    hipError_t e = arena_acquire(g->dp_arena, bytes, st, &base);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(EMO_ERR_OUT_OF_MEMORY, "scratch of %zu bytes: %s", bytes, hipGetErrorString(e));
    }
    dp_layout(S, R, P, &b, static_cast<char *>(base));
    // dp[0] = {P_0}, expanded into the first stage's candidates (row buffer 1 holds P_0)
    e = emo::dp_launch_default_row(b.rows[1], P, F, st);
    if (e == hipSuccess) s = evaluate(g, b.rows[1], 1, b.T, b.E, nullptr, 0, 0, nullptr, nullptr, nullptr, st);
    if (e == hipSuccess && s == EMO_OK)
        e = emo::dp_launch_seed(b.rows[1], P, F, P > 0 ? order[0] : -1, b.T, b.E, b.rows[0], b.state,
                                b.keys[0], b.Tst, b.keys[1], NB, st);
    int64_t cur = 1;
    int kfin = 0;
    // stage i sets pack order[i]: its candidates are in rows[i % 2], its source keys in
    // keys[i % 2], its buckets go to keys[1 - i % 2]
    for (int32_t i = 0; i < P && NB > 0 && e == hipSuccess && s == EMO_OK; ++i) {
        const int x = i % 2;
        const int64_t B = cur * F;
        s = evaluate(g, b.rows[x], B, b.T, b.E, nullptr, 0, 0, nullptr, nullptr, nullptr, st);
        if (s != EMO_OK) break;
        e = emo::dp_launch_bucket(b.T, b.E, b.keys[x], B, F, latency_target, q, bmin, NB, b.keys[1 - x], st);
        if (e == hipSuccess)
            e = emo::dp_launch_advance(b.rows[x], b.T, b.keys[1 - x], NB, P, F, i + 1 < P ? order[i + 1] : -1,
                                       b.rows[1 - x], b.state, b.Tst, b.keys[x], st);
        kfin = 1 - x;
        cur = NB;
    }
    if (e == hipSuccess && s == EMO_OK)
        e = emo::dp_launch_final(b.state, b.keys[kfin], b.Tst, cur, P, latency_target, q, best_levels, result, st);
    hipError_t er = arena_release(g->dp_arena, st);
    if (s != EMO_OK) return s;
    if (e == hipSuccess) e = er;
    return after_launch(e, "emo_dp_search");
}

}  // extern "C"
