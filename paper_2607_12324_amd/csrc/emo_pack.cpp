// Dependency-aware greedy kernel packing (Sec. IV-D, Eq. 5) and the contraction of a per-kernel
// execution graph into its packed graph.  Host-only load-time passes: nothing here touches the
// GPU, so they run on machines without one.
//
// Both passes work on the graph form emo_load_graph takes, where every GPU compute kernel is its
// own input pack.  Graph walks use a canonical topological order (depth, then id), computed here
// with Kahn's algorithm; completion times of Eq. 5 are the all-maximum schedule (level F-1) in
// double precision, so every decision is exact for fp32 inputs.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <unordered_map>
#include <vector>

#include "emo.h"
#include "emo_internal.h"

namespace {

emo_status fail(emo_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    return emo::report(s, buf);
}

bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.f; }

// Deduplicated adjacency in both directions plus the canonical order.
struct Dag {
    int32_t V = 0;
    std::vector<int32_t> src, dst;                 // unique edges, sorted by (src, dst)
    std::vector<int32_t> pred_off, pred, succ_off, succ;
    std::vector<int32_t> order, pos;               // canonical order and each node's place in it
};

emo_status build_dag(int32_t V, int32_t E, const int32_t *edge_src, const int32_t *edge_dst, Dag &d) {
    d.V = V;
    std::vector<int64_t> keys(E);
    for (int32_t i = 0; i < E; ++i) {
        if (edge_src[i] < 0 || edge_src[i] >= V || edge_dst[i] < 0 || edge_dst[i] >= V)
            return fail(EMO_ERR_INVALID_ARGUMENT, "edge %d (%d -> %d) out of range", i, edge_src[i], edge_dst[i]);
        if (edge_src[i] == edge_dst[i]) return fail(EMO_ERR_CYCLE, "self-loop on node %d", edge_src[i]);
        keys[i] = int64_t(edge_src[i]) * V + edge_dst[i];
    }
    std::sort(keys.begin(), keys.end());
    keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
    const size_t m = keys.size();
    d.src.resize(m);
    d.dst.resize(m);
    d.pred_off.assign(V + 1, 0);
    d.succ_off.assign(V + 1, 0);
    for (size_t i = 0; i < m; ++i) {
        d.src[i] = int32_t(keys[i] / V);
        d.dst[i] = int32_t(keys[i] % V);
        d.succ_off[d.src[i] + 1]++;
        d.pred_off[d.dst[i] + 1]++;
    }
    for (int32_t v = 0; v < V; ++v) {
        d.succ_off[v + 1] += d.succ_off[v];
        d.pred_off[v + 1] += d.pred_off[v];
    }
    d.succ.resize(m);
    d.pred.resize(m);
    std::vector<int32_t> fs(d.succ_off.begin(), d.succ_off.end() - 1);
    std::vector<int32_t> fp(d.pred_off.begin(), d.pred_off.end() - 1);
    for (size_t i = 0; i < m; ++i) {
        d.succ[fs[d.src[i]]++] = d.dst[i];
        d.pred[fp[d.dst[i]]++] = d.src[i];
    }
    // Kahn's algorithm for depths (longest path in edges), then a stable bucket sort by depth
    std::vector<int32_t> indeg(V), queue, depth(V, 0);
    queue.reserve(V);
    for (int32_t v = 0; v < V; ++v) {
        indeg[v] = d.pred_off[v + 1] - d.pred_off[v];
        if (indeg[v] == 0) queue.push_back(v);
    }
    for (size_t h = 0; h < queue.size(); ++h) {
        const int32_t v = queue[h];
        for (int32_t j = d.succ_off[v]; j < d.succ_off[v + 1]; ++j) {
            const int32_t u = d.succ[j];
            depth[u] = std::max(depth[u], depth[v] + 1);
            if (--indeg[u] == 0) queue.push_back(u);
        }
    }
    if (int32_t(queue.size()) != V)
        return fail(EMO_ERR_CYCLE, "the graph has a cycle (%d of %d nodes are orderable)", int(queue.size()), int(V));
    int32_t maxd = 0;
    for (int32_t v = 0; v < V; ++v) maxd = std::max(maxd, depth[v]);
    std::vector<int32_t> start(size_t(maxd) + 2, 0);
    for (int32_t v = 0; v < V; ++v) start[depth[v] + 1]++;
    for (int32_t k = 0; k <= maxd; ++k) start[k + 1] += start[k];
    d.order.resize(V);
    d.pos.resize(V);
    for (int32_t v = 0; v < V; ++v) {
        d.pos[v] = start[depth[v]]++;
        d.order[d.pos[v]] = v;
    }
    return EMO_OK;
}

// Shared argument checks; `tables` also checks pack_energy when it is given.
emo_status check_graph(int32_t V, int32_t E, const int32_t *edge_src, const int32_t *edge_dst,
                       const int32_t *node_pack, const float *node_duration, int32_t P, int32_t F,
                       const float *pack_time, const float *pack_energy, std::vector<int32_t> &node_of) {
    if (V < 0 || E < 0 || P < 0) return fail(EMO_ERR_INVALID_ARGUMENT, "negative size");
    if (F < 1 || F > 256) return fail(EMO_ERR_INVALID_ARGUMENT, "num_levels %d outside [1, 256]", F);
    if (P > V) return fail(EMO_ERR_INVALID_ARGUMENT, "more packs (%d) than nodes (%d)", P, V);
    if (E > 0 && (!edge_src || !edge_dst)) return fail(EMO_ERR_INVALID_ARGUMENT, "edge arrays are NULL");
    if (V > 0 && (!node_pack || !node_duration)) return fail(EMO_ERR_INVALID_ARGUMENT, "node arrays are NULL");
    if (P > 0 && !pack_time) return fail(EMO_ERR_INVALID_ARGUMENT, "pack_time is NULL");
    if (int64_t(P) * F > (int64_t(1) << 28)) return fail(EMO_ERR_INVALID_ARGUMENT, "tables too large");
    node_of.assign(P, -1);
    for (int32_t v = 0; v < V; ++v) {
        const int32_t p = node_pack[v];
        if (p < -1 || p >= P) return fail(EMO_ERR_INVALID_ARGUMENT, "node %d has pack id %d outside [-1, %d)", v, p, P);
        if (p >= 0) {
            if (node_of[p] >= 0) return fail(EMO_ERR_INVALID_ARGUMENT, "pack %d appears on more than one node", p);
            node_of[p] = v;
        } else if (!finite_nonneg(node_duration[v])) {
            return fail(EMO_ERR_INVALID_ARGUMENT, "node %d duration must be finite and >= 0", v);
        }
    }
    for (int32_t p = 0; p < P; ++p)
        if (node_of[p] < 0) return fail(EMO_ERR_INVALID_ARGUMENT, "pack %d is on no node", p);
    for (int64_t i = 0; i < int64_t(P) * F; ++i)
        if (!finite_nonneg(pack_time[i]) || (pack_energy && !finite_nonneg(pack_energy[i])))
            return fail(EMO_ERR_INVALID_ARGUMENT, "table entry %lld must be finite and >= 0", (long long)i);
    return EMO_OK;
}

}  // namespace

extern "C" {

emo_status emo_pack_kernels(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                            const int32_t *edge_dst, const int32_t *node_pack,
                            const float *node_duration, const int32_t *node_stream,
                            int32_t num_packs, int32_t num_levels, const float *pack_time,
                            float max_pack_duration, int32_t *pack_group, int32_t *num_groups) {
    const int32_t V = num_nodes, P = num_packs, F = num_levels;
    if (!num_groups || (P > 0 && !pack_group)) return fail(EMO_ERR_INVALID_ARGUMENT, "output pointers are NULL");
    if (V > 0 && !node_stream) return fail(EMO_ERR_INVALID_ARGUMENT, "node_stream is NULL");
    if (std::isnan(max_pack_duration) || !(max_pack_duration > 0.f))
        return fail(EMO_ERR_INVALID_ARGUMENT, "max_pack_duration must be > 0");
    std::vector<int32_t> node_of;
    emo_status s = check_graph(V, num_edges, edge_src, edge_dst, node_pack, node_duration, P, F,
                               pack_time, nullptr, node_of);
    if (s != EMO_OK) return s;
    for (int32_t v = 0; v < V; ++v) {
        if (node_stream[v] < -1) return fail(EMO_ERR_INVALID_ARGUMENT, "node %d has stream %d < -1", v, node_stream[v]);
        if (node_pack[v] >= 0 && node_stream[v] < 0)
            return fail(EMO_ERR_INVALID_ARGUMENT, "kernel node %d has no stream", v);
    }
    Dag d;
    if ((s = build_dag(V, num_edges, edge_src, edge_dst, d)) != EMO_OK) return s;

    // all-maximum completion times and critical predecessors (Eq. 5: the first maximal
    // predecessor in the canonical order)
    auto dur_max = [&](int32_t v) -> double {
        const int32_t p = node_pack[v];
        return p >= 0 ? double(pack_time[size_t(p) * F + (F - 1)]) : double(node_duration[v]);
    };
    std::vector<double> eft(V, 0.0);
    std::vector<int32_t> cpred(V, -1);
    for (int32_t v : d.order) {
        double st = 0.0;
        int32_t best = -1;
        for (int32_t j = d.pred_off[v]; j < d.pred_off[v + 1]; ++j) {
            const int32_t k = d.pred[j];
            if (best < 0 || eft[k] > eft[best] || (eft[k] == eft[best] && d.pos[k] < d.pos[best])) best = k;
        }
        if (best >= 0) st = eft[best];
        cpred[v] = best;
        eft[v] = st + dur_max(v);
    }
    auto same_stream = [&](int32_t a, int32_t b) { return node_stream[a] >= 0 && node_stream[a] == node_stream[b]; };
    // rule 2 per node: every critical successor shares the node's stream
    std::vector<uint8_t> succ_safe(V, 1);
    for (int32_t w = 0; w < V; ++w)
        if (cpred[w] >= 0 && !same_stream(w, cpred[w])) succ_safe[cpred[w]] = 0;

    struct Open { int32_t group, last; double duration; };
    std::unordered_map<int32_t, Open> open;
    const double limit = double(max_pack_duration);
    int32_t groups = 0;
    for (int32_t v : d.order) {
        const int32_t p = node_pack[v];
        if (p < 0) continue;
        const double t_v = dur_max(v);
        auto it = open.find(node_stream[v]);
        bool joins = false;
        if (it != open.end()) {
            const Open &o = it->second;
            bool adjacent = false;
            for (int32_t j = d.pred_off[v]; j < d.pred_off[v + 1] && !adjacent; ++j) adjacent = d.pred[j] == o.last;
            const bool r1 = cpred[v] >= 0 && same_stream(v, cpred[v]);
            const bool r2 = succ_safe[o.last] != 0;
            const bool r3 = o.duration + t_v < limit;
            joins = adjacent && r1 && r2 && r3;
        }
        if (joins) {
            Open &o = it->second;
            pack_group[p] = o.group;
            o.last = v;
            o.duration += t_v;
        } else {
            pack_group[p] = groups;
            open[node_stream[v]] = Open{groups, v, t_v};
            ++groups;
        }
    }
    *num_groups = groups;
    return emo::report(EMO_OK, "");
}

emo_status emo_contract_packs(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                              const int32_t *edge_dst, const int32_t *node_pack,
                              const float *node_duration, int32_t num_packs, int32_t num_levels,
                              const float *pack_time, const float *pack_energy,
                              const int32_t *pack_group, int32_t num_groups, int32_t *packed_node,
                              int32_t *packed_node_pack, float *packed_node_duration,
                              int32_t *packed_src, int32_t *packed_dst, float *group_time,
                              float *group_energy, int32_t *counts) {
    const int32_t V = num_nodes, P = num_packs, F = num_levels, G = num_groups;
    if (!counts) return fail(EMO_ERR_INVALID_ARGUMENT, "counts is NULL");
    if (P > 0 && (!pack_energy || !pack_group)) return fail(EMO_ERR_INVALID_ARGUMENT, "pack arrays are NULL");
    if (V > 0 && (!packed_node || !packed_node_pack || !packed_node_duration))
        return fail(EMO_ERR_INVALID_ARGUMENT, "packed node arrays are NULL");
    if (num_edges > 0 && (!packed_src || !packed_dst)) return fail(EMO_ERR_INVALID_ARGUMENT, "packed edge arrays are NULL");
    if (G < 0 || G > P || (P > 0 && G == 0)) return fail(EMO_ERR_INVALID_ARGUMENT, "num_groups %d outside [1, %d]", G, P);
    if (G > 0 && (!group_time || !group_energy)) return fail(EMO_ERR_INVALID_ARGUMENT, "group tables are NULL");
    std::vector<int32_t> node_of;
    emo_status s = check_graph(V, num_edges, edge_src, edge_dst, node_pack, node_duration, P, F,
                               pack_time, pack_energy, node_of);
    if (s != EMO_OK) return s;
    for (int32_t p = 0; p < P; ++p)
        if (pack_group[p] < 0 || pack_group[p] >= G)
            return fail(EMO_ERR_INVALID_ARGUMENT, "pack %d has group %d outside [0, %d)", p, pack_group[p], G);
    Dag d;
    if ((s = build_dag(V, num_edges, edge_src, edge_dst, d)) != EMO_OK) return s;

    // members of each group in canonical order: first and last kernel
    std::vector<int32_t> first(G, -1), last(G, -1), count(G, 0);
    for (int32_t v : d.order) {
        if (node_pack[v] < 0) continue;
        const int32_t g = pack_group[node_pack[v]];
        if (first[g] < 0) first[g] = v;
        last[g] = v;
        count[g]++;
    }
    for (int32_t g = 0; g < G; ++g)
        if (!count[g]) return fail(EMO_ERR_INVALID_ARGUMENT, "group %d has no member", g);
    // packed nodes: non-kernel nodes and each group's first kernel, by increasing id
    std::vector<int32_t> id(V, -1);
    int32_t n = 0;
    for (int32_t v = 0; v < V; ++v) {
        const int32_t p = node_pack[v];
        if (p < 0 || first[pack_group[p]] == v) {
            id[v] = n;
            packed_node_pack[n] = p < 0 ? -1 : pack_group[p];
            packed_node_duration[n] = p < 0 ? node_duration[v] : 0.f;
            ++n;
        }
    }
    for (int32_t v = 0; v < V; ++v) {
        const int32_t p = node_pack[v];
        packed_node[v] = p < 0 ? id[v] : id[first[pack_group[p]]];
    }
    // surviving dependencies: out of a non-kernel node or a group's last kernel, into a
    // non-kernel node or a group's first kernel
    std::vector<int64_t> keys;
    keys.reserve(d.src.size());
    for (size_t i = 0; i < d.src.size(); ++i) {
        const int32_t a = d.src[i], b = d.dst[i];
        const int32_t pa = node_pack[a], pb = node_pack[b];
        if (pa >= 0 && last[pack_group[pa]] != a) continue;
        if (pb >= 0 && first[pack_group[pb]] != b) continue;
        const int32_t ra = packed_node[a], rb = packed_node[b];
        if (ra != rb) keys.push_back(int64_t(ra) * n + rb);
    }
    std::sort(keys.begin(), keys.end());
    keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
    for (size_t i = 0; i < keys.size(); ++i) {
        packed_src[i] = int32_t(keys[i] / n);
        packed_dst[i] = int32_t(keys[i] % n);
    }
    // group tables: member sums in member order, accumulated in double
    std::vector<double> st(size_t(G) * F, 0.0), se(size_t(G) * F, 0.0);
    for (int32_t v : d.order) {
        const int32_t p = node_pack[v];
        if (p < 0) continue;
        const size_t g = size_t(pack_group[p]);
        for (int32_t f = 0; f < F; ++f) {
            st[g * F + f] += double(pack_time[size_t(p) * F + f]);
            se[g * F + f] += double(pack_energy[size_t(p) * F + f]);
        }
    }
    for (size_t i = 0; i < st.size(); ++i) {
        group_time[i] = float(st[i]);
        group_energy[i] = float(se[i]);
    }
    counts[0] = n;
    counts[1] = int32_t(keys.size());
    return emo::report(EMO_OK, "");
}

}  // extern "C"
