/*
 * emo_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU oracle for EMO's what-if evaluation of DVFS frequency policies over an
 * execution graph (paper: "EMO: Energy Efficiency Modeling and Optimization for AI Workloads",
 * Sec. IV-C and Sec. IV-F).  It is used only by the test suite, by the smoke check and by the
 * benchmark's CPU-baseline leg.  It shares no code with the HIP library and must never be
 * linked into it.
 *
 * Arithmetic: every time and energy is held in double precision (the fp32 inputs convert
 * exactly); no blocking, fusion or reordering beyond the definitions below.
 *
 * Definitions followed (all citations are to the paper):
 *   - completion time C_v = t_v + max over predecessors of C_k            (Eq. 1)
 *     with sources starting at time 0 (the paper leaves comp[pred[v]] undefined for a
 *     node without predecessors; start 0 is the reading taken here);
 *   - makespan T = max_v C_v, energy E = sum_v e_v + E_idle               (Eq. 2)
 *     with E_idle read as static_power * T;
 *   - frequency-dependent cost: a pack's duration and energy come from its latency/energy
 *     tables at the level its policy assigns; other nodes keep their fixed duration and
 *     contribute no energy                                                (Eq. 3, Alg. 1);
 *   - one level per pack (the per-pack form of the policy of Eq. 4);
 *   - the prediction itself is one traversal in topological order that tracks each node's
 *     critical predecessor with a strict "greater than" test               (Alg. 1, Eq. 5);
 *   - slack: total float of the critical-path method, LFT(v) - EFT(v) with
 *     LFT(v) = T for a node without successors, else min over successors (LFT(u) - t_u);
 *     the paper defines slack as the time windows in which a kernel is off the critical path
 *     (Sec. I);
 *   - feasibility T <= T_set and the argmin of energy over feasible policies (Eq. 4), ties
 *     broken by the lower candidate index;
 *   - canonical topological order: nodes sorted by (depth, id), depth(v) = 0 for a source
 *     and 1 + max depth of its predecessors otherwise, computed by memoised recursion.
 *
 * Every function is pinned by the CPU tests (brute force over paths, closed forms, a
 * hand-worked example and invariants); none is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_BAD_ARGUMENT 1
#define ORACLE_CYCLE 2
#define ORACLE_NO_MEMORY 3

typedef struct {
    int V, E, P, F;
    const int *src, *dst;      /* [E] */
    const int *pack;           /* [V] pack id or -1 */
    const float *dur;          /* [V] fixed durations */
    const float *tt, *te;      /* [P*F] latency / energy tables */
    double static_power;
    /* derived adjacency (owned) */
    int *pred_off, *pred;      /* CSR of predecessors */
    int *succ_off, *succ;      /* CSR of successors */
    int *order;                /* canonical topological order */
    int *depth;
} ograph;

static void ograph_free(ograph *g) {
    free(g->pred_off); free(g->pred); free(g->succ_off); free(g->succ);
    free(g->order); free(g->depth);
    memset(g, 0, sizeof(*g));
}

static int build_csr(int V, int E, const int *from, const int *to, int **off_out, int **adj_out) {
    int *off = (int *)calloc((size_t)V + 1, sizeof(int));
    int *adj = (int *)malloc(((size_t)E + 1) * sizeof(int));
    int *fill = (int *)calloc((size_t)V + 1, sizeof(int));
    if (!off || !adj || !fill) { free(off); free(adj); free(fill); return ORACLE_NO_MEMORY; }
    for (int i = 0; i < E; ++i) off[to[i] + 1]++;
    for (int v = 0; v < V; ++v) off[v + 1] += off[v];
    for (int i = 0; i < E; ++i) { int v = to[i]; adj[off[v] + fill[v]++] = from[i]; }
    free(fill);
    *off_out = off; *adj_out = adj;
    return ORACLE_OK;
}

/* depth(v) = 0 without predecessors, else 1 + max over predecessors; memoised recursion
 * written with an explicit stack so that long chains do not overflow the C stack.
 * state: 0 = unvisited, 1 = on the stack, 2 = done. A back edge to a node on the stack is a
 * cycle. */
static int compute_depths(ograph *g) {
    int V = g->V;
    char *state = (char *)calloc((size_t)V + 1, 1);
    int *stack = (int *)malloc(((size_t)V + 1) * sizeof(int));
    int *next = (int *)malloc(((size_t)V + 1) * sizeof(int));
    if (!state || !stack || !next) { free(state); free(stack); free(next); return ORACLE_NO_MEMORY; }
    int rc = ORACLE_OK;
    for (int root = 0; root < V && rc == ORACLE_OK; ++root) {
        if (state[root] == 2) continue;
        int sp = 0;
        stack[sp++] = root; state[root] = 1; next[root] = g->pred_off[root];
        while (sp > 0) {
            int v = stack[sp - 1];
            if (next[v] < g->pred_off[v + 1]) {
                int k = g->pred[next[v]++];
                if (state[k] == 1) { rc = ORACLE_CYCLE; break; }
                if (state[k] == 0) { state[k] = 1; next[k] = g->pred_off[k]; stack[sp++] = k; }
            } else {
                int d = 0;
                for (int i = g->pred_off[v]; i < g->pred_off[v + 1]; ++i) {
                    int dk = g->depth[g->pred[i]] + 1;
                    if (dk > d) d = dk;
                }
                g->depth[v] = d;
                state[v] = 2;
                --sp;
            }
        }
    }
    free(state); free(stack); free(next);
    return rc;
}

static const int *g_sort_depth;
static int cmp_depth_id(const void *a, const void *b) {
    int x = *(const int *)a, y = *(const int *)b;
    if (g_sort_depth[x] != g_sort_depth[y]) return g_sort_depth[x] < g_sort_depth[y] ? -1 : 1;
    return x < y ? -1 : (x > y);
}

static int ograph_init(ograph *g, int V, int E, const int *src, const int *dst, const int *pack,
                       const float *dur, int P, int F, const float *tt, const float *te,
                       double static_power) {
    memset(g, 0, sizeof(*g));
    if (V < 0 || E < 0 || P < 0 || F < 1) return ORACLE_BAD_ARGUMENT;
    for (int i = 0; i < E; ++i) {
        if (src[i] < 0 || src[i] >= V || dst[i] < 0 || dst[i] >= V) return ORACLE_BAD_ARGUMENT;
        if (src[i] == dst[i]) return ORACLE_CYCLE;
    }
    for (int v = 0; v < V && pack; ++v)
        if (pack[v] < -1 || pack[v] >= P) return ORACLE_BAD_ARGUMENT;
    g->V = V; g->E = E; g->P = P; g->F = F;
    g->src = src; g->dst = dst; g->pack = pack; g->dur = dur; g->tt = tt; g->te = te;
    g->static_power = static_power;
    int rc = build_csr(V, E, src, dst, &g->pred_off, &g->pred);
    if (rc == ORACLE_OK) rc = build_csr(V, E, dst, src, &g->succ_off, &g->succ);
    if (rc != ORACLE_OK) { ograph_free(g); return rc; }
    g->order = (int *)malloc(((size_t)V + 1) * sizeof(int));
    g->depth = (int *)malloc(((size_t)V + 1) * sizeof(int));
    if (!g->order || !g->depth) { ograph_free(g); return ORACLE_NO_MEMORY; }
    rc = compute_depths(g);
    if (rc != ORACLE_OK) { ograph_free(g); return rc; }
    for (int v = 0; v < V; ++v) g->order[v] = v;
    g_sort_depth = g->depth;
    qsort(g->order, (size_t)V, sizeof(int), cmp_depth_id);
    return ORACLE_OK;
}

/* Canonical topological order and depths. */
int oracle_topo_order(int V, int E, const int *src, const int *dst, int *order, int *depth) {
    ograph g;
    int rc = ograph_init(&g, V, E, src, dst, NULL, NULL, 0, 1, NULL, NULL, 0.0);
    if (rc != ORACLE_OK) return rc;
    memcpy(order, g.order, (size_t)V * sizeof(int));
    if (depth) memcpy(depth, g.depth, (size_t)V * sizeof(int));
    ograph_free(&g);
    return ORACLE_OK;
}

/* Duration and energy of node v under the level row `lv` (Eq. 3). Sets *bad on a level
 * outside [0, F). */
static void node_cost(const ograph *g, const uint8_t *lv, int v, double *d, double *e, int *bad) {
    int p = g->pack[v];
    if (p < 0) { *d = (double)g->dur[v]; *e = 0.0; return; }
    int l = lv[p];
    if (l >= g->F) { *bad = 1; *d = 0.0; *e = 0.0; return; }
    *d = (double)g->tt[(size_t)p * g->F + l];
    *e = (double)g->te[(size_t)p * g->F + l];
}

/* What-if prediction of one candidate (Alg. 1 with one level per pack):
 * one traversal in topological order; comp[] are completion times, cpred[] critical
 * predecessors (-1: none).  Returns makespan and energy; NaN for both on a bad level. */
static void predict_one(const ograph *g, const uint8_t *lv, double *comp, int *cpred,
                        double *T_out, double *E_out) {
    int bad = 0;
    double Ea = 0.0;
    for (int v = 0; v < g->V; ++v) cpred[v] = -1;
    for (int i = 0; i < g->V; ++i) {
        int v = g->order[i];
        double start = cpred[v] >= 0 ? comp[cpred[v]] : 0.0;
        double d, e;
        node_cost(g, lv, v, &d, &e, &bad);
        comp[v] = start + d;
        Ea += e;
        for (int j = g->succ_off[v]; j < g->succ_off[v + 1]; ++j) {
            int u = g->succ[j];
            if (cpred[u] < 0 || comp[v] > comp[cpred[u]]) cpred[u] = v;
        }
    }
    double T = 0.0;
    for (int v = 0; v < g->V; ++v) if (comp[v] > T) T = comp[v];
    if (bad) { *T_out = NAN; *E_out = NAN; return; }
    *T_out = T;
    *E_out = Ea + g->static_power * T;
}

/* Evaluate B candidates: levels is [B][P] row-major. T and E are [B]. */
int oracle_eval_batch(int V, int E, const int *src, const int *dst, const int *pack,
                      const float *dur, int P, int F, const float *tt, const float *te,
                      double static_power, const uint8_t *levels, int64_t B, double *T,
                      double *En, int nthreads) {
    ograph g;
    int rc = ograph_init(&g, V, E, src, dst, pack, dur, P, F, tt, te, static_power);
    if (rc != ORACLE_OK) return rc;
    int failed = 0;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
    {
        double *comp = (double *)malloc(((size_t)V + 1) * sizeof(double));
        int *cpred = (int *)malloc(((size_t)V + 1) * sizeof(int));
        if (!comp || !cpred) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(static)
            for (int64_t c = 0; c < B; ++c)
                predict_one(&g, levels + (size_t)c * P, comp, cpred, &T[c], &En[c]);
        }
        free(comp); free(cpred);
    }
    ograph_free(&g);
    return failed ? ORACLE_NO_MEMORY : ORACLE_OK;
}

/* Forward completion times, backward latest finish times and slack of every node for one
 * candidate, plus the critical-predecessor array of Alg. 1.  All outputs are [V]. */
int oracle_slack(int V, int E, const int *src, const int *dst, const int *pack, const float *dur,
                 int P, int F, const float *tt, const float *te, double static_power,
                 const uint8_t *lv, double *eft, double *lft, double *slack, int *cpred,
                 double *T_out, double *E_out) {
    ograph g;
    int rc = ograph_init(&g, V, E, src, dst, pack, dur, P, F, tt, te, static_power);
    if (rc != ORACLE_OK) return rc;
    predict_one(&g, lv, eft, cpred, T_out, E_out);
    double T = *T_out;
    int bad = 0;
    for (int i = V - 1; i >= 0; --i) {
        int v = g.order[i];
        double l = T;
        if (g.succ_off[v + 1] > g.succ_off[v]) {
            l = INFINITY;
            for (int j = g.succ_off[v]; j < g.succ_off[v + 1]; ++j) {
                int u = g.succ[j];
                double du, eu;
                node_cost(&g, lv, u, &du, &eu, &bad);
                double lst_u = lft[u] - du;
                if (lst_u < l) l = lst_u;
            }
        }
        lft[v] = l;
        slack[v] = l - eft[v];
    }
    if (bad || isnan(T)) for (int v = 0; v < V; ++v) { lft[v] = NAN; slack[v] = NAN; }
    ograph_free(&g);
    return ORACLE_OK;
}

/* Feasibility (T <= target) and the lowest-energy feasible candidate, lower index on ties.
 * Returns the index, or -1 when no candidate is feasible. */
int64_t oracle_select(const double *T, const double *En, int64_t B, double target,
                      uint8_t *feasible, int64_t *num_feasible) {
    int64_t best = -1, n = 0;
    for (int64_t c = 0; c < B; ++c) {
        int ok = T[c] <= target;   /* false for NaN */
        if (feasible) feasible[c] = (uint8_t)ok;
        if (!ok) continue;
        ++n;
        if (best < 0 || En[c] < En[best]) best = c;
    }
    if (num_feasible) *num_feasible = n;
    return best;
}
