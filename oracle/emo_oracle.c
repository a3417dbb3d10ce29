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
 * Each quantity is computed from its defining equation, one equation per function:
 *   - node cost (Eq. 3): a pack's duration and energy are its latency and energy table entries
 *     at the level its policy assigns (one level per pack, the per-pack form of the policy of
 *     Eq. 4); other nodes keep their fixed duration and use no energy;
 *   - completion time (Eq. 1): C_v = t_v + the largest completion time among v's
 *     predecessors, 0 for a node without predecessors (the paper leaves that maximum
 *     undefined; start 0 is the reading taken here).  Evaluated in a topological order so
 *     that every predecessor is known first;
 *   - makespan and energy (Eq. 2): T = max over all nodes of C_v, E = sum over all nodes of
 *     e_v + E_idle, with E_idle read as static_power * T;
 *   - critical predecessor (Eq. 5): the predecessor of largest completion time; among equal
 *     ones the first in the canonical topological order (the strict comparison with which the
 *     paper's predictor keeps the first one it meets);
 *   - slack: total float of the critical-path method, LFT(v) - C_v with LFT(v) = T for a
 *     node without successors, else the least latest start LFT(u) - t_u over its successors;
 *     the paper describes slack as the time in which a kernel is off the critical path
 *     (Sec. I);
 *   - feasibility T <= T_set and the argmin of energy over feasible policies (Eq. 4), ties
 *     broken by the lower candidate index;
 *   - canonical topological order: nodes sorted by (depth, id), depth(v) = 0 for a source
 *     and 1 + max depth of its predecessors otherwise, computed by memoised recursion.
 * A level byte >= F makes a candidate's makespan, energy and slack NaN (not a policy).
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
    const int *pack;           /* [V] pack id or -1 */
    const float *dur;          /* [V] fixed durations */
    const float *tt, *te;      /* [P*F] latency / energy tables */
    double static_power;
    /* derived adjacency (owned) */
    int *pred_off, *pred;      /* CSR of predecessors */
    int *succ_off, *succ;      /* CSR of successors */
    int *order;                /* canonical topological order */
    int *pos;                  /* position of each node in that order */
    int *depth;
} ograph;

static void ograph_free(ograph *g) {
    free(g->pred_off); free(g->pred); free(g->succ_off); free(g->succ);
    free(g->order); free(g->pos); free(g->depth);
    memset(g, 0, sizeof(*g));
}

/* adjacency lists adj[off[v] .. off[v+1]) = { from[i] : to[i] == v } */
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
    g->pack = pack; g->dur = dur; g->tt = tt; g->te = te;
    g->static_power = static_power;
    int rc = build_csr(V, E, src, dst, &g->pred_off, &g->pred);
    if (rc == ORACLE_OK) rc = build_csr(V, E, dst, src, &g->succ_off, &g->succ);
    if (rc != ORACLE_OK) { ograph_free(g); return rc; }
    g->order = (int *)malloc(((size_t)V + 1) * sizeof(int));
    g->pos = (int *)malloc(((size_t)V + 1) * sizeof(int));
    g->depth = (int *)malloc(((size_t)V + 1) * sizeof(int));
    if (!g->order || !g->pos || !g->depth) { ograph_free(g); return ORACLE_NO_MEMORY; }
    rc = compute_depths(g);
    if (rc != ORACLE_OK) { ograph_free(g); return rc; }
    for (int v = 0; v < V; ++v) g->order[v] = v;
    g_sort_depth = g->depth;
    qsort(g->order, (size_t)V, sizeof(int), cmp_depth_id);
    for (int i = 0; i < V; ++i) g->pos[g->order[i]] = i;
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

/* Eq. 3: dur[v] and en[v] of every node under the level row `lv`.  Returns 0, or 1 when a
 * pack's level lies outside [0, F) (the row is then not a policy). */
static int node_costs(const ograph *g, const uint8_t *lv, double *dur, double *en) {
    int bad = 0;
    for (int v = 0; v < g->V; ++v) {
        int p = g->pack[v];
        if (p < 0) { dur[v] = (double)g->dur[v]; en[v] = 0.0; continue; }
        int l = lv[p];
        if (l >= g->F) { bad = 1; dur[v] = 0.0; en[v] = 0.0; continue; }
        dur[v] = (double)g->tt[(size_t)p * g->F + l];
        en[v] = (double)g->te[(size_t)p * g->F + l];
    }
    return bad;
}

/* Eq. 1: C[v] = dur[v] + max over predecessors k of C[k] (0 without predecessors), taken in
 * topological order so that every C[k] is final when v is reached. */
static void completion_times(const ograph *g, const double *dur, double *C) {
    for (int i = 0; i < g->V; ++i) {
        int v = g->order[i];
        double s = 0.0;
        for (int j = g->pred_off[v]; j < g->pred_off[v + 1]; ++j) {
            int k = g->pred[j];
            if (C[k] > s) s = C[k];
        }
        C[v] = s + dur[v];
    }
}

/* Eq. 2: T = max over nodes of C, E = sum over nodes of e + static_power * T. */
static void makespan_energy(const ograph *g, const double *C, const double *en, double *T_out,
                            double *E_out) {
    double T = 0.0, Ea = 0.0;
    for (int v = 0; v < g->V; ++v) {
        if (C[v] > T) T = C[v];
        Ea += en[v];
    }
    *T_out = T;
    *E_out = Ea + g->static_power * T;
}

/* Eq. 5: cpred[v] = the predecessor of largest completion time, the first in the canonical
 * order among equal ones; -1 for a node without predecessors. */
static void critical_predecessors(const ograph *g, const double *C, int *cpred) {
    for (int v = 0; v < g->V; ++v) {
        int best = -1;
        for (int j = g->pred_off[v]; j < g->pred_off[v + 1]; ++j) {
            int k = g->pred[j];
            if (best < 0 || C[k] > C[best] || (C[k] == C[best] && g->pos[k] < g->pos[best]))
                best = k;
        }
        cpred[v] = best;
    }
}

/* Backward pass of the critical-path method: LFT(v) = T without successors, else the least
 * LFT(u) - dur(u) over successors u, taken in reverse topological order; slack = LFT - C. */
static void total_float(const ograph *g, const double *dur, const double *C, double T,
                        double *lft, double *slack) {
    for (int i = g->V - 1; i >= 0; --i) {
        int v = g->order[i];
        double l = T;
        for (int j = g->succ_off[v]; j < g->succ_off[v + 1]; ++j) {
            int u = g->succ[j];
            double lst_u = lft[u] - dur[u];
            if (j == g->succ_off[v] || lst_u < l) l = lst_u;
        }
        lft[v] = l;
        slack[v] = l - C[v];
    }
}

/* One candidate: costs, completion times, makespan and energy; NaN T and E on a bad level.
 * Returns the bad flag. */
static int evaluate_one(const ograph *g, const uint8_t *lv, double *dur, double *en, double *C,
                        double *T, double *En) {
    int bad = node_costs(g, lv, dur, en);
    completion_times(g, dur, C);
    makespan_energy(g, C, en, T, En);
    if (bad) { *T = NAN; *En = NAN; }
    return bad;
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
        double *buf = (double *)malloc(3 * ((size_t)V + 1) * sizeof(double));
        if (!buf) {
#pragma omp atomic write
            failed = 1;
        } else {
            double *d = buf, *e = buf + V + 1, *C = buf + 2 * ((size_t)V + 1);
#pragma omp for schedule(static)
            for (int64_t c = 0; c < B; ++c)
                evaluate_one(&g, levels + (size_t)c * P, d, e, C, &T[c], &En[c]);
        }
        free(buf);
    }
    ograph_free(&g);
    return failed ? ORACLE_NO_MEMORY : ORACLE_OK;
}

/* Completion times, latest finish times, slack and critical predecessors of every node for one
 * candidate.  All outputs are [V]; a bad level makes lft and slack NaN. */
int oracle_slack(int V, int E, const int *src, const int *dst, const int *pack, const float *dur,
                 int P, int F, const float *tt, const float *te, double static_power,
                 const uint8_t *lv, double *eft, double *lft, double *slack, int *cpred,
                 double *T_out, double *E_out) {
    ograph g;
    int rc = ograph_init(&g, V, E, src, dst, pack, dur, P, F, tt, te, static_power);
    if (rc != ORACLE_OK) return rc;
    double *d = (double *)malloc(2 * ((size_t)V + 1) * sizeof(double));
    if (!d) { ograph_free(&g); return ORACLE_NO_MEMORY; }
    double *e = d + V + 1;
    int bad = evaluate_one(&g, lv, d, e, eft, T_out, E_out);
    critical_predecessors(&g, eft, cpred);
    total_float(&g, d, eft, *T_out, lft, slack);
    if (bad) for (int v = 0; v < V; ++v) { lft[v] = NAN; slack[v] = NAN; }
    free(d);
    ograph_free(&g);
    return ORACLE_OK;
}

/* Makespan, energy and slack of B candidates (levels [B][P]).  per_node = 0: S is [B][P],
 * the slack of pack p at S[c*P + p]; per_node = 1: S is [B][V] indexed by node id.  T and E
 * are [B].  A bad level makes the candidate's T, E and slack row NaN. */
int oracle_slack_batch(int V, int E, const int *src, const int *dst, const int *pack,
                       const float *dur, int P, int F, const float *tt, const float *te,
                       double static_power, const uint8_t *levels, int64_t B, int per_node,
                       double *T, double *En, double *S, int nthreads) {
    ograph g;
    int rc = ograph_init(&g, V, E, src, dst, pack, dur, P, F, tt, te, static_power);
    if (rc != ORACLE_OK) return rc;
    int failed = 0;
    const size_t cols = per_node ? (size_t)V : (size_t)P;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
    {
        double *buf = (double *)malloc(5 * ((size_t)V + 1) * sizeof(double));
        if (!buf) {
#pragma omp atomic write
            failed = 1;
        } else {
            const size_t n = (size_t)V + 1;
            double *d = buf, *e = buf + n, *C = buf + 2 * n, *lft = buf + 3 * n, *sl = buf + 4 * n;
#pragma omp for schedule(static)
            for (int64_t c = 0; c < B; ++c) {
                int bad = evaluate_one(&g, levels + (size_t)c * P, d, e, C, &T[c], &En[c]);
                total_float(&g, d, C, T[c], lft, sl);
                double *row = S + (size_t)c * cols;
                for (int v = 0; v < V; ++v) {
                    double s = bad ? NAN : sl[v];
                    if (per_node) row[v] = s;
                    else if (g.pack[v] >= 0) row[g.pack[v]] = s;
                }
            }
        }
        free(buf);
    }
    ograph_free(&g);
    return failed ? ORACLE_NO_MEMORY : ORACLE_OK;
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
