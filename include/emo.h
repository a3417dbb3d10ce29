/*
 * emo.h -- C ABI of an MI355X (gfx950) library for EMO's batched what-if evaluation of DVFS
 * frequency policies over an execution graph.
 *
 * Paper: "EMO: Energy Efficiency Modeling and Optimization for AI Workloads".
 *   The execution graph G = (V, E) and its precedence edges: Sec. IV-C (what-if analysis).
 *   Completion time, makespan and energy: Sec. IV-C, Eq. 1 and Eq. 2.
 *   Frequency-dependent node cost from per-pack latency/energy tables: Eq. 3, Sec. IV-E Eq. 7,
 *   Alg. 1 (packs take T_f/E_f at their frequency, other nodes keep a fixed duration and no
 *   energy).
 *   The constrained problem (minimum energy subject to a latency target): Eq. 4.
 *   Slack (time in which a kernel is off the critical path): Sec. I and Sec. IV-D.
 *
 * Model computed for one candidate policy (one frequency level per pack):
 *   dur(v)  = pack_time[p][l_p]   if node v is pack p, else node_duration[v]
 *   EST(v)  = 0 for a node without predecessors, else max over predecessors k of EFT(k)
 *   EFT(v)  = EST(v) + dur(v)
 *   T       = max over v of EFT(v)                                   (makespan)
 *   E       = sum over packs p of pack_energy[p][l_p] + static_power * T
 *   LFT(v)  = T for a node without successors, else min over successors u of LFT(u) - dur(u)
 *   slack(v)= LFT(v) - EFT(v)
 *   feasible= T <= latency_target
 *   selected= the feasible candidate of least E, the lower index on equal E; -1 if none.
 *
 * Arithmetic is IEEE fp32 with round-to-nearest-even for times, in the order of the recurrence
 * above, except that the cut-segment kernels time the nodes between two cut nodes from the
 * earlier cut and add the segments' spans, and the chain scan kernels (last_kernels 6 and 8)
 * take slack from prefix sums of durations along each chain instead of the backward recurrence
 * (the same values whenever every time sum is exact, emo_graph_info.exact_time_sums); the
 * pack-energy sum is accumulated in fp32 blocks of at most 64 packs added into an fp64 total,
 * then rounded to fp32 (blocks follow the program order in the one-kernel, segmented and
 * interpreting kernels and each chain's window in the chain kernels, so energies from the two
 * groups of kinds agree to that rounding, not bit for bit).
 *
 * Units are the caller's (the tests use microseconds and power units with energy =
 * power * time).  Level F-1 is conventionally the maximum frequency; nothing here depends on it.
 *
 * Memory: "host" pointers are ordinary CPU memory; "device" pointers are device memory of the
 * GPU the graph was loaded on (e.g. a torch CUDA tensor's data_ptr()).  The caller owns every
 * buffer.  Batch calls are asynchronous on `stream` (a hipStream_t; NULL means the default
 * stream): the caller keeps inputs and outputs alive until the stream has completed.  Scratch
 * device memory is kept by each graph handle (and, for emo_select_from_results, per device)
 * and reused: one buffer for each of the first eight streams that call (calls on one stream
 * are ordered by that stream) and one shared by calls from further streams.  It grows with
 * hipMalloc when a call needs more (waiting for the calls still using it) and is freed with
 * the handle, so steady-state calls allocate nothing and never block the host.  Since a
 * stream's buffer is found again by the stream's handle, a stream must have completed the
 * calls made on it before it is destroyed (a new stream may receive the same handle).
 *
 * Errors: every entry point returns an emo_status.  Argument errors that the host can detect
 * (sizes, null pointers, indices, non-finite or negative values, cycles, misaligned buffers)
 * are reported synchronously and nothing is launched.  emo_last_error() returns a message for
 * the last failure on the calling thread.  A level byte >= F in a candidate is not an error:
 * that candidate's makespan, energy and slack are NaN and it is never feasible.
 *
 * Thread safety: a loaded graph is immutable; calls on one handle from several threads or
 * streams are safe.  Calls from the first eight streams use a scratch buffer per stream; calls
 * from further streams share one, so the device runs those one after the other: such a call on
 * a different stream than the previous one first waits (on the device) for that call's
 * kernels.
 */
#ifndef EMO_H
#define EMO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct emo_graph_s *emo_graph_t;

typedef enum {
    EMO_OK = 0,
    EMO_ERR_INVALID_ARGUMENT = 1,
    EMO_ERR_CYCLE = 2,
    EMO_ERR_OUT_OF_MEMORY = 3,
    EMO_ERR_DEVICE = 4,
    EMO_ERR_UNSUPPORTED = 5
} emo_status;

/* Result of a selection (Eq. 4), written to device memory.  24 bytes, 8-byte aligned. */
typedef struct {
    int64_t index;          /* selected candidate, -1 when none is feasible */
    float energy;           /* its energy, NaN when none */
    float makespan;         /* its makespan, NaN when none */
    int64_t num_feasible;   /* number of candidates with makespan <= target */
} emo_selection;

/* Facts about a loaded graph, for callers and tests. */
typedef struct {
    int32_t num_nodes;
    int32_t num_edges;            /* after duplicate edges are merged */
    int32_t num_packs;
    int32_t num_levels;
    int32_t num_dynamic_nodes;    /* packs and nodes with a pack ancestor */
    int32_t num_dynamic_edges;    /* edges between dynamic nodes */
    int32_t eval_slots;           /* finish-time slots the forward pass keeps live at once */
    int32_t max_depth;            /* largest depth (longest path in edges) */
    float const_makespan;         /* largest finish time among candidate-independent nodes */
    int32_t device;               /* device ordinal, -1 for a host-only graph */
    int32_t pack_order_monotone;  /* 1 if the kernels visit packs in increasing pack id */
    int32_t kernel_mode;          /* emo_kernel_mode in effect */
    int32_t specialized;          /* bit 0: specialised eval/select kernels are compiled,
                                     bit 1: specialised slack kernels are compiled,
                                     bit 2: specialisation was tried and failed,
                                     bit 3: segmented kernels are compiled,
                                     bit 4: cut-segment kernels are compiled */
    float compile_seconds;        /* time spent compiling specialised kernels */
    int32_t last_kernels;         /* kernels of the last batch call: 0 interpreted, 1 one
                                     specialised kernel, 2 segmented specialised kernels,
                                     3 chain lanes (one lane per chain and candidate),
                                     4 windowed chain lanes (a wave per chain, 64 candidates;
                                     pack windows staged in LDS; calls without slack), 5 cut
                                     segments (the
                                     segments between cut nodes evaluated in parallel),
                                     6 two-pass chain scan (windowed chain lanes whose slack
                                     comes from a second forward pass; calls with slack), 7
                                     time-interval kernel
                                     specialised to the graph (emo_eval_intervals; 0 there
                                     means the interpreting kernel), 8 two-pass chain scan
                                     whose window copies and slack stores follow per-thread
                                     plans fixed for the call (chain_scan_full) */
    int32_t chain_lanes;          /* lanes per candidate of the chain-lane kernels, 0 when the
                                     candidate-dependent nodes do not form at most 64 disjoint
                                     chains */
    int32_t num_implied_edges;    /* merged edges u -> v that the kernels skip because another
                                     path leads from u to v (they never decide a maximum or a
                                     minimum; results are unchanged) */
    int32_t chain_window;         /* packs per window of the windowed chain-lane kernel, 0 when
                                     it does not apply (more than 16 chains, a chain that goes
                                     back to an earlier window, fewer than 16 packs); calls
                                     without slack use it on graphs that neither one kernel nor
                                     the segmented kernels take, when levels and slack are
                                     16-byte aligned (rows of a
                                     pack count that is not a multiple of 16 are copied from
                                     the dwords around each 16-byte piece) */
    int32_t cut_segments;         /* segments of the cut-segment kernels, 0 when they do not
                                     apply.  A cut node is one that every other node precedes
                                     or follows (an all-stream synchronisation): no path
                                     bypasses it, so its slack is zero and, measured from the
                                     finish time of the cut before them, the finish times and
                                     slack of the nodes between two cuts depend on those
                                     nodes' levels only (Eq. 1; slack as in Sec. III-A:
                                     time off the critical path).  The kernels cut the graph
                                     there, in segments of at most 256 packs, when packs are
                                     visited in increasing id and segments start at multiples
                                     of 32 packs.  Batch calls of graphs too large for one
                                     specialised kernel use them when levels (and slack) are
                                     16-byte aligned and fewer than 2^30 candidates are
                                     evaluated.  They time each segment from its own start, so
                                     their results are those of the other kernels bit for bit
                                     when exact_time_sums is 1, and agree with them to fp32
                                     rounding otherwise. */
    int32_t chain_scan_window;    /* packs per window of the two-pass chain scan kernels
                                     (last_kernels 6 and 8), 0 when it does not apply: the
                                     candidate-dependent nodes must form at most 16 disjoint
                                     chains visiting the windows in increasing order (the
                                     windowed layout); calls with slack use it on graphs of at
                                     least 768 steps (the segmented kernels, slower there, take
                                     161-767) when levels and slack are 16-byte aligned */
    int32_t chain_scan_full;      /* 1 when slack calls of the two-pass chain scan run the
                                     kernel with per-thread copy plans (last_kernels 8): every
                                     window lies wholly inside the graph (P a multiple of
                                     chain_scan_window), a thread holds at most four 16-byte
                                     pieces of a window's slack tile (at least
                                     chain_scan_window / 16 chains) and a workgroup's slack
                                     rows span less than 4 GiB; 0 otherwise */
    int32_t hip_runtime_version;  /* hipRuntimeGetVersion of the HIP runtime the library runs
                                     on (e.g. 70051831 for 7.0.51831).  The run-time compiler
                                     of the specialised kernels is the hiprtc of that same
                                     runtime, so this also names the compiler that builds
                                     them. */
    int32_t exact_time_sums;      /* 1 when every time value (table times, fixed durations) is
                                     a multiple of one power of two u and the sum of all
                                     nodes' largest durations is below 2^24 u: every sum and
                                     difference of times along paths is then exact in fp32 in
                                     any order, and every kernel kind computes bit-identical
                                     makespans and slack.  0 otherwise: the cut-segment and
                                     chain scan kernels then agree with the others to
                                     rounding. */
} emo_graph_info;

/* Which kernels evaluate a graph.
 *   EMO_KERNELS_AUTO         kernels specialised to the graph (generated and compiled at run
 *                            time on first use) when the graph is small enough, otherwise the
 *                            precompiled interpreting kernels.  Default.
 *   EMO_KERNELS_INTERPRETED  always the precompiled kernels that interpret a compiled program.
 *   EMO_KERNELS_SPECIALIZED  like AUTO, but a failed specialisation is reported as
 *                            EMO_ERR_DEVICE by the batch call instead of falling back.
 * Both kinds compute bit-identical results, except that the cut-segment and chain scan kernels
 * round differently on graphs whose time sums are not exact (emo_graph_info.exact_time_sums
 * 0) and that chain kernels group the energy sum by chain windows (see the arithmetic above). */
typedef enum {
    EMO_KERNELS_AUTO = 0,
    EMO_KERNELS_INTERPRETED = 1,
    EMO_KERNELS_SPECIALIZED = 2
} emo_kernel_mode;

/*
 * Load an execution graph and its pack tables (Sec. IV-C; the inputs of Alg. 1).
 *   num_nodes, num_edges  V >= 0, E >= 0.
 *   edge_src, edge_dst    host int32 [E]: node edge_src[i] finishes before edge_dst[i] starts.
 *                         Duplicates are merged.  A self-loop or cycle gives EMO_ERR_CYCLE.
 *   node_pack             host int32 [V]: pack id in [0, P) or -1 for a fixed node.  Every pack
 *                         id in [0, P) must appear on exactly one node.
 *   node_duration         host float [V]: duration of fixed nodes, finite and >= 0 (ignored on
 *                         pack nodes).
 *   num_packs, num_levels P >= 0 packs, 1 <= F <= 256 frequency levels.
 *   pack_time, pack_energy host float [P*F], row-major by pack: latency and energy of pack p at
 *                         level l at index p*F + l; finite and >= 0.
 *   static_power          finite, >= 0: energy per unit time charged over the makespan (the
 *                         idle-energy term of Eq. 2 / Alg. 1).
 *   device                GPU ordinal to hold the graph, or -1 for a host-only graph (analysis
 *                         and emo_graph_topo_order only; batch calls then fail with
 *                         EMO_ERR_UNSUPPORTED).
 *   out                   receives the handle; the library deep-copies every input.
 */
emo_status emo_load_graph(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                          const int32_t *edge_dst, const int32_t *node_pack,
                          const float *node_duration, int32_t num_packs, int32_t num_levels,
                          const float *pack_time, const float *pack_energy, float static_power,
                          int32_t device, emo_graph_t *out);

/* Release a graph and its device memory.  NULL is accepted.  Work still queued on a stream
 * that uses the graph must have completed. */
emo_status emo_free_graph(emo_graph_t g);

/* Fill `info` (host). */
emo_status emo_graph_get_info(emo_graph_t g, emo_graph_info *info);

/* Choose the kernels used by later batch calls on `g` (an emo_kernel_mode).  Not to be called
 * while batch calls on `g` may run concurrently on another thread. */
emo_status emo_graph_set_kernel_mode(emo_graph_t g, int32_t mode);

/*
 * Canonical topological order (the traversal order of Alg. 1): nodes sorted by depth, then by
 * node id, where depth is 0 for a node without predecessors and 1 + the largest predecessor
 * depth otherwise.  order: host int32 [V]; depth: host int32 [V] or NULL.
 */
emo_status emo_graph_topo_order(emo_graph_t g, int32_t *order, int32_t *depth);

/*
 * Makespan and energy of B candidate policies (Eq. 1-3, Alg. 1 with one level per pack).
 *   levels    device uint8 [B][P], row-major by candidate: level of pack p in candidate c at
 *             c*P + p.
 *   B         0 <= B < 2^32; B = 0 is a no-op.
 *   makespan  device float [B];  energy  device float [B].  Either may be NULL.
 */
emo_status emo_eval_policies(emo_graph_t g, const uint8_t *levels, int64_t num_candidates,
                             float *makespan, float *energy, void *stream);

/*
 * Slack of every pack (per_node = 0) or of every node (per_node = 1) for B candidates: the
 * forward pass above followed by a backward pass in reverse topological order.
 *   slack     device float, [B][P] indexed by pack id, or [B][V] indexed by node id.
 *   makespan, energy  optional device float [B] outputs of the same forward pass (NULL to skip).
 */
emo_status emo_slack(emo_graph_t g, const uint8_t *levels, int64_t num_candidates, float *slack,
                     int32_t per_node, float *makespan, float *energy, void *stream);

/*
 * Evaluate B candidates and select the least-energy one whose makespan is <= latency_target
 * (Eq. 4 over the given candidate batch), ties to the lower index.
 *   feasible_mask  device uint32 [ceil(B/32)] or NULL: bit (c % 32) of word c / 32 is set iff
 *                  candidate c is feasible.
 *   result         device emo_selection, 8-byte aligned, written once at the end of the call
 *                  (one partial record per workgroup goes to stream-ordered scratch memory and a
 *                  single-workgroup kernel reduces them; there are no global atomics).
 */
emo_status emo_select_policy(emo_graph_t g, const uint8_t *levels, int64_t num_candidates,
                             float latency_target, uint32_t *feasible_mask,
                             emo_selection *result, void *stream);

/*
 * The whole hot path in one pass over the candidates, as one kernel launch (plus, with
 * `result`, a one-workgroup kernel that completes the selection): makespan and energy
 * (Eq. 1-3), slack of every
 * pack or node when `slack` is given, and the feasibility mask and least-energy feasible
 * candidate under `latency_target` (Eq. 4) when `feasible_mask` or `result` is given.
 * Every output is optional (NULL); their layouts are those of emo_eval_policies, emo_slack and
 * emo_select_policy.  latency_target is ignored without mask and result.
 */
emo_status emo_evaluate(emo_graph_t g, const uint8_t *levels, int64_t num_candidates,
                        float *makespan, float *energy, float *slack, int32_t per_node,
                        float latency_target, uint32_t *feasible_mask, emo_selection *result,
                        void *stream);

/*
 * emo_evaluate with several latency targets in the same pass (Eq. 4 once per target over one
 * evaluation of the batch, e.g. the operating points of a latency sweep): the evaluating kernel
 * writes every target's mask bits and selection partial records, and one finalize launch with a
 * workgroup per target completes every selection.  Each target's mask and result are those
 * emo_evaluate gives for that target alone, bit for bit.
 *   num_targets      1 <= n <= 8.
 *   latency_targets  host float [n], none NaN (checked when a mask or the results are given).
 *   feasible_masks   host array of n device pointers (each device uint32 [ceil(B/32)] or NULL),
 *                    or NULL for no masks.
 *   results          device emo_selection [n], 8-byte aligned, or NULL: results[k] is target k's
 *                    selection.
 * makespan, energy, slack and per_node as in emo_evaluate.  The scratch for the partial records
 * (n x 16 bytes per evaluating workgroup) comes from the graph's stream-ordered arena.
 */
emo_status emo_evaluate_targets(emo_graph_t g, const uint8_t *levels, int64_t num_candidates,
                                float *makespan, float *energy, float *slack, int32_t per_node,
                                int32_t num_targets, const float *latency_targets,
                                uint32_t *const *feasible_masks, emo_selection *results,
                                void *stream);

/*
 * The same selection from makespans and energies already computed (e.g. a second latency
 * target over one evaluation).  makespan, energy: device float [B].
 */
emo_status emo_select_from_results(const float *makespan, const float *energy,
                                   int64_t num_candidates, float latency_target,
                                   uint32_t *feasible_mask, emo_selection *result, void *stream);

/*
 * emo_select_from_results without any allocation, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, outputs and results as emo_select_from_results.  Its selection partial
 * records (16 bytes per 1024 candidates) live in a static 4 MiB device array that each GPU the
 * library runs on holds until the process ends; the call allocates and frees nothing.  The
 * first call on a device looks up that device's address of the array (hipGetSymbolAddress).
 *   num_candidates  0 <= B <= 268,435,456 (2^28, the records the array holds); a larger B is
 *                   EMO_ERR_INVALID_ARGUMENT and launches nothing.
 * Every call on one GPU shares that GPU's array (nothing in it needs to start cleared: each
 * call writes every record it reads).  Calls that overlap on one GPU (on different streams
 * with no ordering between them, or from several threads) race on it and may return a wrong
 * selection; calls ordered on one stream are safe.
 */
emo_status emo_select_from_results_noalloc(const float *makespan, const float *energy,
                                           int64_t num_candidates, float latency_target,
                                           uint32_t *feasible_mask, emo_selection *result,
                                           void *stream);

/*
 * Time-interval frequency policies: the general policy form P = {<T_i, F_i>} of the optimisation
 * problem (Sec. IV-A) as Alg. 1 evaluates it.  The batch shares K = num_intervals intervals
 * [T_i, T_{i+1}) with T_0 = 0, T_i = change_points[i - 1] and the last interval open-ended; each
 * candidate gives one level per interval.  A pack runs at the level of the interval that holds
 * its start time (the largest finish time among its predecessors, 0 for a source; half-open
 * intervals, so a start equal to a change point takes the later interval), which makes a pack's
 * level depend on the schedule.  makespan as in Eq. 1-2; energy = the packs' table energies plus
 * the idle energy of Alg. 1, read as idle_power[F_i] times the wall time interval i covers
 * inside [0, makespan) (with idle_power[f] = the graph's static_power for every f, one interval
 * gives the energy of emo_eval_policies with that level on every pack).  The graph's
 * static_power is not used here.
 *   levels:        device uint8 [B][K], row-major (16-byte aligned rows with K % 16 == 0 are
 *                  read as vectors; any layout works).  A byte >= F anywhere in a row makes
 *                  that candidate's makespan and energy NaN (never feasible).
 *   num_intervals: K in [1, 256].
 *   change_points: host float [K - 1] (NULL when K = 1), finite, > 0, strictly increasing;
 *                  copied at the call (the kernel receives them as arguments).
 *   idle_power:    host float [F], finite, >= 0 (power units; times are in microseconds).
 *   makespan, energy: device float [B] or NULL; feasible_mask, result and latency_target as in
 *                  emo_evaluate.
 * Asynchronous on `stream`; invalid arguments are reported synchronously and launch nothing.
 */
emo_status emo_eval_intervals(emo_graph_t g, const uint8_t *levels, int64_t num_candidates,
                              int32_t num_intervals, const float *change_points,
                              const float *idle_power, float *makespan, float *energy,
                              float latency_target, uint32_t *feasible_mask,
                              emo_selection *result, void *stream);

/* Profiling hook: while set, batch calls on `g` record `begin_event` on their stream right
 * before the kernel that evaluates the candidates and `end_event` right after it (before the
 * single-workgroup kernel that completes a selection).  Both are hipEvent_t handles (NULL
 * disables); the caller owns them.  Not to be called while batch calls on `g` may run
 * concurrently on another thread. */
emo_status emo_graph_set_timing_events(emo_graph_t g, void *begin_event, void *end_event);

/*
 * Near-optimal policy search (Alg. 2, Sec. IV-F) with one frequency interval per pack, on the
 * device.  Dynamic programming over the packs in `pack_order`: dp[0] holds the all-maximum
 * policy P_0 (level F-1 everywhere); stage i sets pack order[i] to every level f in every
 * stored policy, evaluates those policies with the batch evaluator (Alg. 1), drops the ones
 * whose makespan exceeds latency_target, and keeps for each makespan bucket
 * floor(makespan / quantum) the one of least energy (among equal energies the first in the
 * order (stored policy by increasing bucket, level f increasing)).  The result is the least
 * energy over the last stage's policies (among equal energies the lowest bucket).  Makespans
 * and energies are the evaluator's fp32 values; buckets are computed in double precision.
 *   latency_target   T_max, finite (the constraint of Eq. 4).
 *   quantum          bucket width, finite and > 0 (the paper discretises time at e.g. 1 ms).
 *   pack_order       host int32 [P], a permutation of the pack ids, or NULL for 0..P-1.
 *   max_states       the most buckets the search may keep: from one below the bucket of the
 *                    least possible makespan (every pack at its fastest level) to the bucket of
 *                    latency_target; a larger range is EMO_ERR_INVALID_ARGUMENT (choose a
 *                    coarser quantum).  Device scratch grows with max_states x F x P bytes.
 *   best_levels      device uint8 [P]: the policy found; left unchanged when none is found.
 *   result           device emo_selection, 8-byte aligned: index = floor(makespan / quantum) of
 *                    the policy found, or -1 (energy and makespan NaN) when no policy meets
 *                    the target; num_feasible = the policies stored after the last stage.
 * One call runs P + 1 evaluations of at most max_states x F candidates each, asynchronously on
 * `stream`.  Not to be called concurrently with itself on the same graph.
 */
emo_status emo_dp_search(emo_graph_t g, float latency_target, float quantum, const int32_t *pack_order,
                         int32_t max_states, uint8_t *best_levels, emo_selection *result, void *stream);

/*
 * Dependency-aware greedy kernel packing (Sec. IV-D: the critical predecessor of Eq. 5, the two
 * dependency-safety rules and the granularity rule), a host-only load-time pass that needs no
 * GPU.  The input is a graph in emo_load_graph's form whose packs are single GPU compute
 * kernels, plus the stream of every node.  Completion times are the all-maximum schedule
 * (level F-1 everywhere, in double precision); the critical predecessor of a node is its
 * predecessor of latest completion, the first in the canonical topological order among equals,
 * and the critical successors of u are the nodes whose critical predecessor is u.  Kernels are
 * visited in the canonical topological order; each stream has one open pack.  Kernel v joins
 * the open pack of its stream when that pack's last kernel u is a direct predecessor of v and
 *   rule 1: v and its critical predecessor are on the same stream,
 *   rule 2: every critical successor of u is on u's stream,
 *   rule 3: the pack's duration at level F-1 plus v's (summed in double) < max_pack_duration;
 * otherwise v opens a new pack.  Groups are numbered in the order of their first kernels.
 *   edges, node_pack, node_duration, tables: host arrays as in emo_load_graph (pack_energy is
 *                  not needed here); every pack must sit on exactly one node.
 *   node_stream:   host int32 [V]: the GPU stream of each node, >= 0 for every kernel (pack)
 *                  node; -1 for host or other nodes that are on no stream.
 *   max_pack_duration: the granularity bound (the paper uses 5 ms), > 0; +inf disables it.
 *   pack_group:    host int32 [P] out: the group (new pack) of each input pack.
 *   num_groups:    host out: the number of groups.
 * Synchronous.  Invalid arguments give EMO_ERR_INVALID_ARGUMENT, a cycle EMO_ERR_CYCLE, and
 * leave the outputs unspecified.
 */
emo_status emo_pack_kernels(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                            const int32_t *edge_dst, const int32_t *node_pack,
                            const float *node_duration, const int32_t *node_stream,
                            int32_t num_packs, int32_t num_levels, const float *pack_time,
                            float max_pack_duration, int32_t *pack_group, int32_t *num_groups);

/*
 * The packed graph of a grouping of the packs (Sec. IV-D: a pack keeps the incoming
 * dependencies of its first kernel and the outgoing dependencies of its last; the ones in
 * between are dropped), in emo_load_graph's form, host-only.  A group's members are ordered by
 * the canonical topological order.  Packed nodes are the non-kernel nodes and one node per
 * group, numbered by increasing id of the input node standing for them (for a group, its first
 * kernel).  An input edge a -> b survives as packed_node[a] -> packed_node[b] when a is a
 * non-kernel node or its group's last kernel, b is a non-kernel node or its group's first
 * kernel, and the two packed nodes differ; duplicates are merged, edges come out sorted by
 * (src, dst).  A group's latency and energy at level f are the sums of its members' entries,
 * accumulated in double in member order and rounded to fp32.
 *   pack_group, num_groups: as produced by emo_pack_kernels (any grouping in [0, num_groups)
 *                  with no empty group is accepted).
 *   packed_node:   host int32 [V] out: the packed node standing for each input node.
 *   packed_node_pack, packed_node_duration: host [V] capacity, out: the packed graph's
 *                  node_pack (the group id, or -1) and node_duration (0 for groups).
 *   packed_src, packed_dst: host int32 [E] capacity, out: the packed graph's edges.
 *   group_time, group_energy: host float [num_groups * F] out, row-major.
 *   counts:        host int32 [2] out: packed nodes, packed edges.
 * Synchronous; errors as in emo_pack_kernels.
 */
emo_status emo_contract_packs(int32_t num_nodes, int32_t num_edges, const int32_t *edge_src,
                              const int32_t *edge_dst, const int32_t *node_pack,
                              const float *node_duration, int32_t num_packs, int32_t num_levels,
                              const float *pack_time, const float *pack_energy,
                              const int32_t *pack_group, int32_t num_groups, int32_t *packed_node,
                              int32_t *packed_node_pack, float *packed_node_duration,
                              int32_t *packed_src, int32_t *packed_dst, float *group_time,
                              float *group_energy, int32_t *counts);

/*
 * Microbenchmark pack model (Sec. IV-E, Eq. 6-7), a host-only load-time pass that needs no GPU.
 * For every pack p, the non-negative weights x = argmin ||B x - b_p||^2 subject to x >= 0 over
 * the microbenchmark suite (Eq. 6), then the pack's tables at every level f:
 *   pack_time[p][f] = sum_i x_i bench_time[i][f],  pack_energy[p][f] = sum_i x_i bench_energy[i][f]
 * (Eq. 7), accumulated in double in benchmark order and rounded to fp32: the tables
 * emo_load_graph takes.  The solver is Lawson and Hanson's active-set method with Householder
 * QR on the passive columns, in double precision.  When B has full column rank the minimiser is
 * unique; otherwise (fewer metrics than benchmarks) the residual is, and the weights are one
 * minimiser.
 *   metric_matrix: host float [n][m] row-major: metric r of benchmark i at the default
 *                  frequency (n = num_metrics >= 1, m = num_benchmarks in [1, 64]), finite.
 *   bench_time, bench_energy: host float [m][F], finite, >= 0; F = num_levels in [1, 256].
 *   pack_metrics:  host float [P][n]: each pack's metric vector b_p at the default frequency.
 *   weights:       host float [P][m] out, or NULL.
 *   pack_time, pack_energy: host float [P][F] out.
 *   num_threads:   host threads to use (packs are independent); <= 0 for all cores.
 * Synchronous.  EMO_ERR_INVALID_ARGUMENT for bad sizes, NULLs or non-finite inputs;
 * EMO_ERR_UNSUPPORTED if a pack's iteration does not converge (outputs then unspecified).
 */
emo_status emo_pack_model(int32_t num_metrics, int32_t num_benchmarks, const float *metric_matrix,
                          int32_t num_levels, const float *bench_time, const float *bench_energy,
                          int32_t num_packs, const float *pack_metrics, float *weights,
                          float *pack_time, float *pack_energy, int32_t num_threads);

/* Diagnostics: the HIP source of the kernels specialised to `g` (the text EMO_KERNELS_AUTO
 * compiles on first use), NUL-terminated.  With buf == NULL, *len receives the size needed
 * including the NUL; otherwise at most *len bytes are written.  Works on host-only graphs.
 * EMO_ERR_UNSUPPORTED when the graph is too large for one specialised kernel. */
emo_status emo_graph_specialized_source(emo_graph_t g, char *buf, int64_t *len);

/* Diagnostics: the HIP source of the segmented specialised kernels of `g`, used for calls
 * without slack on graphs too large for one kernel or whose (time, energy) table exceeds the
 * 64 KB one kernel holds in LDS, and for slack on graphs too large to keep every finish time in
 * registers: one
 * forward kernel per segment of consecutive steps, launched in order, then one backward kernel
 * per segment in reverse order, which recomputes finish times from checkpointed values instead
 * of reading stored ones.  Same buffer convention as emo_graph_specialized_source.
 * EMO_ERR_UNSUPPORTED when the graph uses no segmented kernels. */
emo_status emo_graph_segmented_source(emo_graph_t g, char *buf, int64_t *len);

/* Diagnostics: the HIP source of the cut-segment kernels of `g` (see cut_segments in
 * emo_graph_info): segment kernels whose grid row y evaluates one segment for a group of
 * candidates (four segments per kernel; forward only, and forward with slack), launched one
 * after another, and the kernel that adds up the segments' makespans and energy blocks and
 * completes the selection.  Same buffer convention as
 * emo_graph_specialized_source.  EMO_ERR_UNSUPPORTED when the graph has no cut segments. */
emo_status emo_graph_cut_source(emo_graph_t g, char *buf, int64_t *len);

/* Diagnostics: the HIP source of the time-interval kernel specialised to `g` (what
 * emo_eval_intervals compiles on first use when the graph is small enough for one specialised
 * kernel): emo_iv, whose workgroups copy their candidates' rows into LDS with coalesced loads and
 * find each pack's interval in a bucket table of the change points (in dynamic LDS, with the
 * rows).  Same buffer convention as emo_graph_specialized_source.  EMO_ERR_UNSUPPORTED when the
 * graph is too large for one kernel. */
emo_status emo_graph_interval_source(emo_graph_t g, char *buf, int64_t *len);

/* Static string naming a status code. */
const char *emo_status_string(emo_status s);

/* Message describing the last failure on the calling thread ("" if none). */
const char *emo_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EMO_H */
