// Internal interface between the host side of the library (graph analysis, program
// compilation, argument checking) and the HIP kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "emo.h"

namespace emo {

// Records `message` as the calling thread's last error (clears it for EMO_OK); returns `s`.
emo_status report(emo_status s, const char *message);

constexpr int kTablePad = 256;   // extra zeroed table entries: any level byte stays in bounds

// Slot references of the interpreting kernels.  A finish time (forward) or latest start time
// (backward) that is read again soon lives in a 32-entry register bank of each lane ("hot",
// indexed wave-uniformly); one that stays live longer lives in device scratch laid out
// [slot][candidate] ("cold", bit 31 of the reference set).
constexpr uint32_t kColdRef = 0x80000000u;
constexpr int kHotSlots = 32;
constexpr uint32_t kStepSink = 1u;   // forward: the node has no successor
constexpr uint32_t kStepOut = 2u;    // the step writes its value to `out`

// Forward step (32 bytes, one scalar load): a candidate-dependent node in topological order.
struct FwdStep {
    int32_t pack;       // pack id, or -1 for a node of fixed duration
    uint32_t cst;       // fp32 bits: latest finish among candidate-independent predecessors
    uint32_t dur;       // fp32 bits: the fixed duration (pack == -1)
    uint32_t flags;     // kStepSink | kStepOut
    uint32_t out;       // slot reference of the finish time
    int32_t in_begin;   // predecessor references: ins[in_begin, in_begin + in_count)
    int32_t in_count;
    int32_t pad;
};

// Backward step (32 bytes), in reverse order of the forward steps.
struct BwdStep {
    int32_t pack;       // pack id, or -1
    uint32_t dur;       // fp32 bits: the fixed duration (pack == -1)
    uint32_t flags;     // kStepOut: predecessors read this node's latest start time
    uint32_t out;       // slot reference of the latest start time
    int32_t succ_begin; // successor references: succs[succ_begin, succ_begin + succ_count)
    int32_t succ_count; // 0 for a sink: its latest finish is the makespan
    int32_t col;        // slack output column, -1 for none
    int32_t fwd;        // index of the node's forward step (its finish time is kept there)
};

// A compiled traversal for the interpreting kernels.
struct DevProgram {
    int32_t n_ops = 0;
    int32_t n_cold = 0;          // cold forward slots
    int32_t n_cold_bwd = 0;      // cold backward slots
    float t_const = 0.f;         // makespan floor from candidate-independent nodes
    int32_t monotone = 1;        // packs visited in increasing id
    const FwdStep *fwd = nullptr;
    const uint32_t *ins = nullptr;
    const BwdStep *bwd = nullptr;     // slack programs only
    const uint32_t *succs = nullptr;
};

struct DevGraph {
    int32_t V = 0, P = 0, F = 1;
    float static_power = 0.f;
    const float2 *tab = nullptr;   // [P*F + kTablePad] interleaved (time, energy)
    const float *tabt = nullptr;   // [P*F + kTablePad] times only (backward passes)
    DevProgram eval;               // forward over candidate-dependent nodes
    DevProgram slack_pack;         // forward + backward over candidate-dependent nodes
    DevProgram slack_node;         // forward + backward over every node
};

// Selection partial records: one per block of the evaluating kernel, reduced by
// launch_select_finalize (16 bytes each: least key, feasible count, makespan).
constexpr size_t kPartialBytes = 16;

// The latency targets of one evaluation, passed to the kernels by value (the layout of the
// kernels' EmoTargets): target k's feasibility mask to mask[k] (when not NULL) and its partial
// records to part + k * nparts * kPartialBytes (all targets, when part is not NULL).  n = 0: no
// mask and no selection.
constexpr int kMaxTargets = 8;
struct SelTargets {
    int32_t n = 0;
    int32_t pad = 0;
    int64_t nparts = 0;
    void *part = nullptr;
    float t[kMaxTargets] = {};
    uint32_t *mask[kMaxTargets] = {};
};
static_assert(sizeof(SelTargets) == 120, "kernel argument layout of the targets");
// One target (the single-target entry points): none when neither mask nor part is given.
inline SelTargets one_target(float target, uint32_t *mask, void *part, int64_t nparts) {
    SelTargets tg;
    if (mask || part) {
        tg.n = 1;
        tg.t[0] = target;
        tg.mask[0] = mask;
        tg.part = part;
        tg.nparts = nparts;
    }
    return tg;
}

// Interpreting kernels.  T, E, mask, part may each be NULL; `part` receives one selection
// partial record per block (forward_blocks(B) of them).
// Device scratch (bytes) the interpreting kernels need for B candidates: cold slots, and for
// slack the forward finish times kept for the backward pass.  The caller passes that much
// (256-byte aligned) as `scratch`.
size_t forward_scratch_bytes(const DevProgram &prog, int64_t B);
size_t slack_scratch_bytes(const DevProgram &prog, int64_t B);
hipError_t launch_forward(const DevGraph &g, const uint8_t *levels, int64_t B, float *T, float *E,
                          const SelTargets &tg, void *scratch, hipStream_t s);
hipError_t launch_slack(const DevGraph &g, const DevProgram &prog, int32_t out_cols,
                        const uint8_t *levels, int64_t B, float *slack, float *T, float *E,
                        const SelTargets &tg, void *scratch, hipStream_t s);
int64_t forward_blocks(int64_t B);

// A time-interval policy batch (the policy form of Sec. IV-A; Alg. 1): K intervals [T_i,
// T_{i+1}) with T_0 = 0 and the last one open-ended; each candidate's row holds K levels.  Passed
// to the kernel by value (2 KB of kernel arguments).
// pack energies are summed in fp32 blocks of this many packs (program order) added into fp64
constexpr int kEnergyBlock = 64;
constexpr int kMaxIntervals = 256;
constexpr int kMaxLevels = 256;
struct IvPolicy {
    int32_t K = 1;
    float pts[kMaxIntervals - 1];   // change points T_1 < ... < T_{K-1}
    float idle[kMaxLevels];         // idle power per level
};
// Makespan, energy and the selection stage 1 of B interval policies (forward_blocks(B) partials);
// scratch as for launch_forward (forward_scratch_bytes(g.eval, B)).
hipError_t launch_intervals(const DevGraph &g, const IvPolicy &pol, const uint8_t *levels, int64_t B,
                            float *T, float *E, const SelTargets &tg, void *scratch, hipStream_t s);
hipError_t launch_empty_result(emo_selection *res, hipStream_t s);
// Stage 2 for every target of tg with part: results[k] from target k's records.
hipError_t launch_select_finalize(const SelTargets &tg, emo_selection *results, hipStream_t s);
// Stage 1 of a selection from stored makespans and energies (select_results_blocks(B)
// partials: one per 1024 candidates).
int64_t select_results_blocks(int64_t B);
// The static selection scratch of emo_select_from_results_noalloc: the largest batch its
// records cover, and the current device's address of it (looked up once per device).
constexpr int kNoAllocMaxDevices = 64;
int64_t noalloc_max_candidates();
hipError_t noalloc_scratch(int dev, void **out);
// (tg.nparts must be select_results_blocks(B))
hipError_t launch_select_results(const float *T, const float *E, int64_t B, const SelTargets &tg,
                                 hipStream_t s);

// ---------------------------------------------------------------- chain-lane kernels

// Graphs whose candidate-dependent steps form disjoint chains (at most one candidate-dependent
// predecessor and successor each): one lane per chain and candidate.
constexpr int kChainStepBlock = 8;    // steps per unrolled block (and per backward checkpoint)
struct ChainStep {                    // 16 bytes
    int32_t pack;                     // pack id, or -1 (fixed node or padding)
    float cst;                        // latest finish among candidate-independent predecessors
    float dur;                        // fixed duration (pack == -1); 0 for padding
    int32_t pad;
};
// Step record of the windowed layout: the chain's steps in pack window w (packs
// [w*win, (w+1)*win)).
struct ChainWinStep {                 // 16 bytes
    uint32_t ct;                      // col | (col * F) << 16, col = pack id - w*win, or win for
                                      // a fixed node (or a no-op step)
    float cst;                        // latest finish among candidate-independent predecessors
    float dur;                        // fixed duration; 0 for a pack
    uint32_t pad;
};
struct DevChains {
    int32_t lanes = 0;                // lanes per candidate: a power of two in [1, 64]
    int32_t lane_log = 0;
    int32_t len = 0;                  // steps per chain, padded to a multiple of kChainStepBlock
    float t_const = 0.f;              // makespan floor from candidate-independent nodes
    const ChainStep *steps = nullptr; // [len][lanes]
    const int32_t *pos = nullptr;     // [P]: step * lanes + chain of each pack
    // windowed layout (win > 0): one block of blk_bytes per window: hdr_words int32 (chain c's
    // steps are records hdr[c] .. hdr[c+1]-1), then the window's ChainWinStep records: 8 no-op
    // steps, each chain's steps padded with no-op steps to a multiple of 4, chain after chain,
    // 8 no-op steps; it exists when every chain visits the windows in increasing order
    int32_t nc = 0;                   // chains
    int32_t win = 0;                  // packs per window, a power of two in [16, 256]
    int32_t nwin = 0;
    int32_t groups = 0;               // groups of 64 candidates per workgroup
    int32_t fixed = 0;                // 1 if some step is a fixed node
    int32_t hdr_words = 0;            // nc + 1 rounded up to a multiple of 4
    int32_t blk_bytes = 0;
    const uint4 *blocks = nullptr;    // [nwin][blk_bytes / 16]
    // every window lies wholly inside the graph (P a multiple of win), a thread of the windowed
    // kernel holds at most four float4 pieces of the slack tile, and a workgroup's slack rows
    // span less than 2^32 bytes: the second-pass kernel with per-thread copy plans applies
    int32_t full = 0;
};
// Whether the windowed kernel's LDS working set and prefetch fit for `nc` chains, F levels,
// windows of W packs and step blocks of blk_bytes (rows16: P is a multiple of 16); sets the
// candidate groups per workgroup.
bool chain_window_fits(int32_t nc, int32_t F, int32_t W, int32_t blk_bytes, bool rows16, int32_t *groups);
// Whether a call runs the windowed kernel (the layout exists and the buffers are 16-byte
// aligned).
bool chains_windowed_ok(const DevChains &c, const uint8_t *levels, const float *slack);
// Whether a call runs the windowed kernel with slack from a second forward pass (a call with
// slack on the windowed layout, buffers 16-byte aligned).
bool chains_scan_ok(const DevChains &c, const uint8_t *levels, const float *slack);
// Whether that call runs the second-pass kernel with per-thread copy plans (chains_scan_full).
bool chains_scan_full_ok(const DevChains &c, const uint8_t *levels, const float *slack);
// Scratch of launch_chains: backward checkpoints and chain-ordered slack (slack only), and
// makespan/energy buffers.
size_t chains_scratch_bytes(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                            const float *slack);
// Makespan/energy (and per-pack slack when `slack`); the selection stage 1 runs from the stored
// makespans and energies (select_results_blocks(B) partial records in `part`).
hipError_t launch_chains(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                         float *T, float *E, float *slack, const SelTargets &tg, void *scratch,
                         hipStream_t s);

// ---------------------------------------------------------------- policy search (Alg. 2)

// Kernels of emo_dp_search (one frequency interval per pack).  dp_launch_seed stores P_0 (row0,
// evaluated) and expands it into the first stage's F candidate rows.  A stage: the batch
// evaluator computes the makespans and energies of its S*F candidate rows, dp_launch_bucket
// keeps for each of the NB buckets (floor(makespan / q) - bmin) the least key (fp32 energy
// bits << 32 | candidate) among the candidates that come from a stored state (src_keys not
// empty) and meet tmax, and dp_launch_advance writes each bucket's winner as the next stage's
// candidate rows (level f at p_next), or after the last stage as a stored state with its
// makespan, and clears the stage's source keys for the next bucket step.
hipError_t dp_launch_default_row(uint8_t *row, int32_t P, int32_t F, hipStream_t s);
hipError_t dp_launch_seed(const uint8_t *row0, int32_t P, int32_t F, int32_t p, const float *T,
                          const float *E, uint8_t *rows, uint8_t *state, unsigned long long *key,
                          float *Tst, unsigned long long *out_keys, int64_t NB, hipStream_t s);
hipError_t dp_launch_bucket(const float *T, const float *E, const unsigned long long *src_keys,
                            int64_t B, int32_t F, float tmax, double q, int64_t bmin, int64_t NB,
                            unsigned long long *keys, hipStream_t s);
hipError_t dp_launch_advance(const uint8_t *rows, const float *T, const unsigned long long *keys,
                             int64_t NB, int32_t P, int32_t F, int32_t p_next, uint8_t *next_rows,
                             uint8_t *state, float *Tst, unsigned long long *done_keys, hipStream_t s);
// The least-energy stored state with makespan <= tmax (ties: lowest bucket) to best and res.
hipError_t dp_launch_final(const uint8_t *states, const unsigned long long *keys, const float *Tst,
                           int64_t S, int32_t P, float tmax, double q, uint8_t *best,
                           emo_selection *res, hipStream_t s);

// ---------------------------------------------------------------- graph-specialised kernels

// One candidate-dependent node of the graph in traversal order.
struct JitOp {
    int32_t pack;                  // pack id or -1
    float cst;                     // start-time floor from candidate-independent predecessors
    float dur;                     // fixed duration (pack == -1)
    std::vector<int32_t> in;       // steps of candidate-dependent predecessors
    std::vector<int32_t> out;      // steps of successors (all candidate-dependent)
};

struct JitGraph {
    int32_t P = 0, F = 1;
    float static_power = 0.f;
    float t_const = 0.f;
    bool pack_monotone = true;
    std::vector<JitOp> ops;
};

// Level words are read a line at a time only when packs are visited in increasing id; in any
// other order a word would stay live from its first to its last use (register pressure), so each
// level byte is then loaded on its own.
inline int jit_level_width(const JitGraph &g) {
    if (!g.pack_monotone) return 1;
    return g.P % 16 == 0 ? 16 : (g.P % 4 == 0 ? 4 : 1);
}

// Segmented specialised kernels, for graphs too large for one straight-line kernel: the steps
// are cut into segments, each with a forward kernel and (for slack) a backward kernel; the
// forward kernels run in order, then the backward kernels in reverse order, on one stream.
// Values crossing a kernel boundary go through device scratch rows [row][bp] (bp = the padded
// grid size).  A backward kernel does not read stored finish times: it recomputes them one
// sub-segment at a time from the checkpointed inputs of that sub-segment.
struct ChainPlan {
    std::vector<int32_t> seg;       // segment boundaries in steps: seg[0] = 0 < ... < seg[m] = n
    std::vector<int32_t> sub;       // recompute sub-segment boundaries (a refinement of seg)
    std::vector<int32_t> ck_row;    // checkpoint row of f_i, or -1
    std::vector<char> ck_always;    // that row is also read by a later forward kernel
    std::vector<int32_t> bk_row;    // row of s_i (latest start) read by an earlier segment, or -1
    int32_t n_ck = 0, n_bk = 0;
    bool slack = false;
    bool staged = false;            // slack written through LDS as 128-byte lines (16-byte stores)
    int block = 256;                // workgroup of the forward kernels
    int bblock = 512;               // workgroup of the backward kernels
    int segments() const { return static_cast<int>(seg.size()) - 1; }
};

// Scratch layout of one chained evaluation (floats unless noted), each [rows][bp] with the
// pitch bp = chain_pitch(B):
//   ck [n_ck], bk [n_bk], Tc (makespan so far) [1], Ebc (open fp32 energy block) [1],
//   Edc (fp64 energy sum) [1, doubles]
inline int64_t chain_pitch(int64_t B) { return (B + 63) / 64 * 64; }
size_t chain_scratch_bytes(const ChainPlan &cp, int64_t B);

// Cut-segment kernels, for graphs with cut steps: steps that every other node of the graph
// precedes or follows (an all-stream synchronisation, for instance).  No path bypasses a cut,
// so a cut step is on every longest path and has zero slack; measured from the finish time of
// the cut before it, the finish times, latest start times and slack of the steps between two
// cuts depend on those steps' levels only.  With every duration a multiple of one power of two
// u and the sum of all nodes' largest durations below 2^24 u, each of these values is an exact
// fp32 number however the additions are ordered, so the segments are evaluated independently
// and in parallel (one kernel, one grid row per segment), each writing its local makespan and
// its energy blocks; a last kernel adds them up in order (makespan, energy, selection) and
// overwrites the slack rows of candidates with an invalid level with NaN.  A segment kernel
// takes a few segments (grid rows); compile time grows faster than linearly with the code of
// one kernel, so the segments are spread over several kernels.
struct CutPlan {
    std::vector<int32_t> seg;       // segment boundaries in steps: seg[0] = 0 < ... < seg[m] = n;
                                    // every segment but possibly the last ends with a cut step
    bool closed_last = true;        // the last segment ends with a cut step as well
    std::vector<int32_t> sub;       // recompute sub-segments of the slack kernel (refine seg)
    std::vector<int32_t> blk0;      // first energy block row of each segment; blk0[m] = rows
    std::vector<char> ck;           // f_i is read by a later sub-segment of its segment
    int block = 512;                // workgroup of the segment kernels and the finishing kernel
    int per_kernel = 4;             // segments per slack segment kernel (grid rows); the kernels
                                    // of consecutive groups of segments run one after another
    int per_kernel_fwd = 16;        // segments per forward-only segment kernel (smaller code: more
                                    // segments per kernel, so that small batches launch fewer)
    int segments() const { return static_cast<int>(seg.size()) - 1; }
    int kernels() const { return (segments() + per_kernel - 1) / per_kernel; }
    int kernels_fwd() const { return (segments() + per_kernel_fwd - 1) / per_kernel_fwd; }
};

// Scratch of a cut-segment evaluation, each [rows][bp] floats with bp = chain_pitch(B):
//   D (local makespan of each segment, NaN for an invalid level) [m], energy blocks [blk0[m]]
size_t cut_scratch_bytes(const CutPlan &cp, int64_t B);

struct JitModule {
    hipModule_t module = nullptr;
    hipFunction_t select = nullptr;  // forward pass with optional outputs and selection
    hipFunction_t slack = nullptr;   // only for graphs small enough to keep every finish time
    double compile_seconds = 0.0;
    int block = 256;
    // resident workgroups of the one-kernel select / slack kernels on the device (their grid,
    // at most one workgroup per group of `block` candidates, so each loads the table once)
    int64_t select_cap = 0, slack_cap = 0;
    // segmented kernels
    bool chain = false;
    ChainPlan plan;
    std::vector<hipFunction_t> cf, cb;   // forward kernel of each segment, backward kernel
    // cut-segment kernels
    bool cut = false;
    CutPlan cut_plan;
    std::vector<hipFunction_t> kf;       // segment kernels, forward only (one per group)
    std::vector<hipFunction_t> ks;       // segment kernels, forward and slack
    hipFunction_t kfin = nullptr;        // makespan, energy, selection, NaN rows
    // time-interval kernel: its static LDS bytes and the device's per-workgroup limit
    int iv_static_lds = 0, iv_max_lds = 0;
};

// Bytes per level load in generated kernels (16, 4 or 1): the alignment they need.

std::string jit_generate(const JitGraph &g, bool with_slack, bool tab_lds, int block);
// Segments of about seg_ops steps (cut where the pack steps so far are a multiple of 64) and
// recompute sub-segments of at most sub_ops steps.
ChainPlan jit_chain_plan(const JitGraph &g, bool with_slack, int seg_ops, int sub_ops);
std::string jit_generate_chain(const JitGraph &g, const ChainPlan &cp);
int jit_compile_chain(const std::string &src, const ChainPlan &cp, JitModule *out, std::string *log);
// Blocks of the segmented kernels' grid (one selection partial each).
int64_t jit_chain_blocks(const JitModule &m, int64_t B);
// Forward kernels (and, with S, the backward kernels) of a chained evaluation.  scratch holds
// chain_scratch_bytes(plan, jit_chain_blocks * block) bytes.
hipError_t jit_launch_chain(const JitModule &m, const uint8_t *levels, int64_t B,
                            const float2 *tab, const float *tabt, void *scratch, float *S,
                            float *T, float *E, const SelTargets &tg, hipStream_t s);
// Plan of the cut-segment kernels over the cut steps `cuts` (increasing step indices): segments
// of whole cut-to-cut pieces with at most max_packs packs each, recompute sub-segments of
// sub_packs packs.  Returns an empty plan (no segments) when a piece is larger.
CutPlan jit_cut_plan(const JitGraph &g, const std::vector<int32_t> &cuts, int max_packs, int sub_packs);
std::string jit_generate_cut(const JitGraph &g, const CutPlan &cp);
int jit_compile_cut(const std::string &src, const CutPlan &cp, JitModule *out, std::string *log);
// Selection partial records of a cut-segment evaluation.
int64_t jit_cut_blocks(const JitModule &m, int64_t B);
// Segment kernel (forward only, or with slack S) and the finishing kernel.  scratch holds
// cut_scratch_bytes(plan, B) bytes.
hipError_t jit_launch_cut(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                          void *scratch, float *S, float *T, float *E, const SelTargets &tg, hipStream_t s);
// 0 on success; otherwise *log holds the compiler's or loader's message.
int jit_compile(const std::string &src, bool with_slack, JitModule *out, std::string *log);
void jit_unload(JitModule *m);
// Candidate groups of the one-kernel specialised kernels for B candidates (one selection
// partial each).
int64_t jit_blocks(const JitModule &m, int64_t B);
// Time-interval kernel specialised to the graph (emo_iv, any K): each workgroup copies its
// candidates' rows to LDS and looks the start times' intervals up in a bucket table; the batch's
// change points, idle powers and bucket table parameters by value.
constexpr int kIvMaxBuckets = 4096;
struct IvJitArgs {
    int32_t K = 1, M = 1;
    float scale = 0.f;
    int32_t pad = 0;
    float pts[kMaxIntervals - 1];
    float idle[kMaxLevels];
};
std::string jit_generate_intervals(const JitGraph &g, bool tab_lds, int block);
int jit_compile_intervals(const std::string &src, JitModule *out, std::string *log);
// Dynamic LDS bytes of emo_iv for K intervals and M buckets (bucket table, then the rows).
size_t jit_iv_dyn_lds(int block, int K, int M);
// Resident workgroups of emo_iv on the current device with that dynamic LDS (0: unknown).
int64_t jit_iv_cap(const JitModule &m, int K, int M);
hipError_t jit_launch_intervals(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                                const IvJitArgs &a, int64_t cap, float *T, float *E, const SelTargets &tg,
                                hipStream_t s);
// Sets select_cap / slack_cap from the occupancy of the compiled kernels (current device).
void jit_set_caps(JitModule *m);
// Forward pass; T, E, mask, part may each be NULL.
hipError_t jit_launch_forward(const JitModule &m, const uint8_t *levels, int64_t B,
                              const float2 *tab, float *T, float *E, const SelTargets &tg, hipStream_t s);
// Forward + backward slack pass with the same optional outputs.
hipError_t jit_launch_slack(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                            float *S, float *T, float *E, const SelTargets &tg, hipStream_t s);

}  // namespace emo
