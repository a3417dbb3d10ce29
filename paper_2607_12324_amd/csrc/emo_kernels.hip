// Precompiled HIP kernels for gfx950: batched what-if evaluation of per-pack frequency
// policies by interpreting a program compiled from the graph (used for graphs too large to
// specialise, for per-node slack and for inputs the specialised kernels cannot take).
//
// Layout: one candidate policy per lane.  Every lane of a wave walks the same program (the
// graph is shared by all candidates), so steps, predecessor lists and slot references are
// wave-uniform and come through scalar loads; only level bytes, the table entries they select
// and finish times differ per lane.
//
// Per forward step (one node in topological order, Eq. 1 and Alg. 1):
//   EST = max(cst, finish times of candidate-dependent predecessors)
//   EFT = EST + dur,  dur = table time at the pack's level (Eq. 3) or the fixed duration
// The makespan is the max over sinks (Eq. 2); pack energies are summed in fp32 blocks of 64
// packs added into an fp64 total, and the static term static_power * T closes Eq. 2.  The
// backward pass (slack) walks the steps in reverse: LFT = min over successors of their latest
// start (T for a sink), slack = LFT - EFT, latest start = LFT - dur.
//
// Storage per lane:
//   hot    32-entry register bank (uniform dynamic index) for values read again soon;
//   cold   device scratch [slot][candidate] for values that stay live long;
//   keep   device scratch [step][candidate]: every finish time, for the backward pass;
//   levels the current 128-byte line of the candidate's level row, in registers.
// Scratch layouts put one wave's access to a slot in one contiguous 256-byte segment.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <cstring>
#include <mutex>

#include "emo_internal.h"
#include "emo_select.h"

// Selection partial records of emo_select_from_results_noalloc, one 16-byte record per group
// of candidates: a static array each device holds until the process ends.  In host code its
// name is not a device address; host code reaches it only through the address that
// hipGetSymbolAddress returns for the current device (emo::noalloc_scratch below).
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace emo {
namespace {

constexpr int kBlock = EMO_BLOCK;
constexpr int kWave = EMO_WAVE;
constexpr int kWavesPerBlock = EMO_WAVES_PER_BLOCK;
constexpr int kStage = 32;            // packs per staged slack segment (one 128-byte line)
constexpr size_t kLdsBudget = 60 * 1024;

typedef float f32x32 __attribute__((ext_vector_type(32)));
typedef unsigned int u32x32 __attribute__((ext_vector_type(32)));

__device__ __forceinline__ uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// Program records and edge lists are never written while a kernel runs.  Reading them through
// the constant address space lets the compiler use scalar loads: a vector load there would be
// followed by a wait that also covers every store still in flight.
#define EMO_CONST_AS __attribute__((address_space(4)))
template <class T>
__device__ __forceinline__ T ld_prog(const T *p, int64_t i) {
    static_assert(sizeof(T) % 4 == 0, "program records are made of 32-bit words");
    const EMO_CONST_AS uint32_t *q = (const EMO_CONST_AS uint32_t *)(p + i);
    uint32_t w[sizeof(T) / 4];
#pragma unroll
    for (int k = 0; k < static_cast<int>(sizeof(T) / 4); ++k) w[k] = q[k];
    T v;
    __builtin_memcpy(&v, w, sizeof(T));
    return v;
}
__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// The candidate's level row, read one 128-byte line (8 x 16 bytes) at a time into a register
// bank `w` (kept as a plain local of the calling pass so that it stays in VGPRs).
struct Row {
    const uint8_t *row;
    int P;
    bool vec;       // rows are 16-byte aligned: line loads; otherwise byte loads
};

__device__ __forceinline__ void load_line(const Row &r, u32x32 &w, int gidx) {
    const uint4 *src = reinterpret_cast<const uint4 *>(r.row) + gidx * 8;
    const int nvec = min(8, (r.P - gidx * 128 + 15) / 16);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        if (k < nvec) {
            const uint4 v = src[k];
            w[4 * k + 0] = v.x;
            w[4 * k + 1] = v.y;
            w[4 * k + 2] = v.z;
            w[4 * k + 3] = v.w;
        }
    }
}

__device__ __forceinline__ unsigned level_at(const Row &r, u32x32 &w, int &group, int p) {
    if (!r.vec) return r.row[p];
    const int gidx = p >> 7;
    if (gidx != group) {
        load_line(r, w, gidx);
        group = gidx;
    }
    const unsigned word = w[(p >> 2) & 31];
    return (word >> ((p & 3) << 3)) & 0xffu;
}

// Table access.  kTabGlobal: straight from device memory; kTabLds: the whole table staged in LDS
// at kernel start; kTabWindow: windows of 2^wlog packs' rows staged into a double-buffered LDS
// area by the workgroup, one barrier per window, the next window prefetched into registers
// while the current one is in use.  Windows need the program to visit packs in increasing id
// (decreasing in the backward pass); every wave of the workgroup walks the same program, so all
// of them reach each window change at the same step.
enum TabMode { kTabGlobal = 0, kTabLds = 1, kTabWindow = 2 };
constexpr int kWindowBytes = 8192;
constexpr int kWindowEntries = kWindowBytes / 8;   // float2 entries per LDS half
static_assert(kWindowBytes == 2 * 16 * kBlock, "two 16-byte pieces of a window per thread");

template <int MODE>
struct Tab {
    const float2 *tab;     // global table, or the whole LDS copy (kTabLds)
    float2 *buf;           // kTabWindow: LDS [2][window entries]
    int F;
    int wlog;              // packs per window = 1 << wlog
    int went;              // table entries per window
    int64_t n_entries;     // valid entries of the global table
    int cur;               // window in use
    float4 pre0, pre1;     // this thread's two pieces of the next window

    // Loads window w's rows into registers.  Indices past the table are clamped to its last
    // piece: those LDS entries belong to packs beyond the last one and are never read.
    __device__ __forceinline__ void fetch(int w) {
        const float4 *src = reinterpret_cast<const float4 *>(tab);
        const int64_t last = n_entries / 2 - 1;
        const int64_t base = static_cast<int64_t>(w < 0 ? 0 : w) * went / 2;
        const int64_t i0 = base + threadIdx.x, i1 = i0 + kBlock;
        pre0 = src[i0 < last ? i0 : last];
        pre1 = src[i1 < last ? i1 : last];
    }
    __device__ __forceinline__ void commit(int w) {
        float4 *dst = reinterpret_cast<float4 *>(buf + (w & 1) * kWindowEntries);
        dst[threadIdx.x] = pre0;
        dst[threadIdx.x + kBlock] = pre1;
    }
    // Makes window w current; dir is +1 in the forward pass, -1 in the backward pass.
    __device__ __forceinline__ void enter(int w, int dir) {
        if (w == cur + dir) {
            commit(w);
        } else {   // first window of a pass (or a jump): stage synchronously
            __syncthreads();
            fetch(w);
            commit(w);
        }
        __syncthreads();
        cur = w;
        fetch(w + dir);
    }
    // The backward pass walks windows downward: refetch the one below the current window.
    __device__ __forceinline__ void turn() {
        if (MODE == kTabWindow) fetch(cur - 1);
    }
    __device__ __forceinline__ float2 get(int pack, int l, int dir) {
        if (MODE != kTabWindow) return tab[pack * F + l];
        const int w = pack >> wlog;
        if (w != cur) enter(w, dir);
        return buf[(w & 1) * kWindowEntries + (pack - (w << wlog)) * F + l];
    }
};

struct Scratch {
    float *cold;        // [n_cold][bpad]
    float *keep;        // [n_ops][bpad] (slack) or nullptr
    float *cold_bwd;    // [n_cold_bwd][bpad]
    int64_t bpad;
    int64_t col;        // this lane's column
};

__device__ __forceinline__ float slot_get(const f32x32 &hot, const float *cold, int64_t bpad,
                                          int64_t col, uint32_t ref) {
    if (ref & kColdRef) return cold[static_cast<int64_t>(ref & ~kColdRef) * bpad + col];
    return hot[ref];
}

__device__ __forceinline__ void slot_set(f32x32 &hot, float *cold, int64_t bpad, int64_t col,
                                         uint32_t ref, float v) {
    if (ref & kColdRef) cold[static_cast<int64_t>(ref & ~kColdRef) * bpad + col] = v;
    else hot[ref] = v;
}

struct Fwd {
    float T;
    float E;
    bool bad;
};

template <int MODE, bool KEEP>
__device__ __forceinline__ Fwd run_forward(const DevProgram &pr, Tab<MODE> &tab, int F, float static_power,
                           const Row &row, f32x32 &hot, const Scratch &sc) {
    u32x32 lw;
    int lgroup = -1;
    float T = pr.t_const;
    double eacc = 0.0;
    float eblk = 0.f;
    int nblk = 0;
    bool bad = false;
    const int n = pr.n_ops;
    for (int i = 0; i < n; ++i) {
        const FwdStep st = ld_prog(pr.fwd, i);
        const uint32_t flags = uni(st.flags);
        const int32_t pack = uni(st.pack);
        const int32_t nin = uni(st.in_count);
        const int32_t ib = uni(st.in_begin);
        float est = __uint_as_float(uni(st.cst));
        for (int j = 0; j < nin; ++j)
            est = fmaxf(est, slot_get(hot, sc.cold, sc.bpad, sc.col, uni(ld_prog(pr.ins, ib + j))));
        float dur;
        if (pack >= 0) {
            unsigned l = level_at(row, lw, lgroup, pack);
            bad |= l >= static_cast<unsigned>(F);
            l = l < static_cast<unsigned>(F) ? l : 0u;
            const float2 te = tab.get(pack, static_cast<int>(l), 1);
            dur = te.x;
            eblk += te.y;
            if (++nblk == kEnergyBlock) {
                eacc += static_cast<double>(eblk);
                eblk = 0.f;
                nblk = 0;
            }
        } else {
            dur = __uint_as_float(uni(st.dur));
        }
        const float eft = est + dur;
        if (flags & kStepOut) slot_set(hot, sc.cold, sc.bpad, sc.col, uni(st.out), eft);
        if (flags & kStepSink) T = fmaxf(T, eft);
        if (KEEP) sc.keep[static_cast<int64_t>(i) * sc.bpad + sc.col] = eft;
    }
    eacc += static_cast<double>(eblk);
    Fwd f;
    f.E = static_cast<float>(eacc + static_cast<double>(static_power) * static_cast<double>(T));
    f.T = T;
    f.bad = bad;
    if (bad) {
        f.T = __builtin_nanf("");
        f.E = __builtin_nanf("");
    }
    return f;
}

// Writes the slack of packs [p0, p0 + kStage) of the wave's 64 candidates, staged in LDS as
// stg[pack - p0][lane] (stride 65 floats), with 16-byte stores: each candidate's segment is one
// 128-byte line.
__device__ __forceinline__ void flush_stage(const float *stg, float *__restrict__ S, int64_t cols,
                                            int64_t wbase, int64_t B, int p0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int lane = threadIdx.x % kWave;
    constexpr int per_row = kStage / 4;
#pragma unroll
    for (int m = 0; m < per_row; ++m) {
        const int j = lane + kWave * m;
        const int r = j / per_row, part = j % per_row;
        float4 v;
        v.x = stg[(4 * part + 0) * 65 + r];
        v.y = stg[(4 * part + 1) * 65 + r];
        v.z = stg[(4 * part + 2) * 65 + r];
        v.w = stg[(4 * part + 3) * 65 + r];
        const int64_t row = wbase + r;
        if (row < B) *reinterpret_cast<float4 *>(S + row * cols + p0 + 4 * part) = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int MODE, bool STAGED>
__device__ __forceinline__ void run_backward(const DevProgram &pr, Tab<MODE> &tab, int F, float T, bool bad,
                             const Row &row, f32x32 &hot, const Scratch &sc, float *__restrict__ S,
                             int64_t cols, int64_t cand, bool active, float *stg, int64_t wbase,
                             int64_t B) {
    u32x32 lw;
    int lgroup = -1;
    tab.turn();
    const int n = pr.n_ops;
    const float inf = __builtin_inff();
    const float nan = __builtin_nanf("");
    const int lane = threadIdx.x % kWave;
    float eft_next = n > 0 ? sc.keep[static_cast<int64_t>(uni(ld_prog(pr.bwd, 0).fwd)) * sc.bpad + sc.col] : 0.f;
    for (int r = 0; r < n; ++r) {
        const BwdStep st = ld_prog(pr.bwd, r);
        const float eft = eft_next;
        if (r + 1 < n)   // the next step's finish time is fetched one step ahead
            eft_next = sc.keep[static_cast<int64_t>(uni(ld_prog(pr.bwd, r + 1).fwd)) * sc.bpad + sc.col];
        const uint32_t flags = uni(st.flags);
        const int32_t pack = uni(st.pack);
        const int32_t ns = uni(st.succ_count);
        const int32_t sb = uni(st.succ_begin);
        const int32_t col = uni(st.col);
        float lft = T;
        if (ns > 0) {
            lft = inf;
            for (int j = 0; j < ns; ++j)
                lft = fminf(lft, slot_get(hot, sc.cold_bwd, sc.bpad, sc.col, uni(ld_prog(pr.succs, sb + j))));
        }
        float dur;
        if (pack >= 0) {
            unsigned l = level_at(row, lw, lgroup, pack);
            l = l < static_cast<unsigned>(F) ? l : 0u;
            dur = tab.get(pack, static_cast<int>(l), -1).x;
        } else {
            dur = __uint_as_float(uni(st.dur));
        }
        if (flags & kStepOut) slot_set(hot, sc.cold_bwd, sc.bpad, sc.col, uni(st.out), lft - dur);
        if (col >= 0) {
            const float v = bad ? nan : lft - eft;
            if (STAGED) {
                stg[(col & (kStage - 1)) * 65 + lane] = v;
                if ((col & (kStage - 1)) == 0) flush_stage(stg, S, cols, wbase, B, col);
            } else if (active) {
                S[cand * cols + col] = v;
            }
        }
    }
}

// Sets up table access for a kernel (stages the whole table when MODE == kTabLds).
template <int MODE>
__device__ __forceinline__ Tab<MODE> make_tab(const DevGraph &g, float4 *smem, int wlog) {
    Tab<MODE> t;
    t.F = g.F;
    t.wlog = wlog;
    t.went = (1 << wlog) * g.F;
    t.n_entries = static_cast<int64_t>(g.P) * g.F + kTablePad;
    t.cur = -2;
    t.buf = nullptr;
    t.tab = g.tab;
    if (MODE == kTabLds) {
        float2 *lds = reinterpret_cast<float2 *>(smem);
        for (int64_t i = threadIdx.x; i < t.n_entries; i += blockDim.x) lds[i] = g.tab[i];
        __syncthreads();
        t.tab = lds;
    } else if (MODE == kTabWindow) {
        t.buf = reinterpret_cast<float2 *>(smem);
    }
    return t;
}

struct LaneCtx {
    int64_t gid, cand, wbase;
    bool active;
};

__device__ __forceinline__ LaneCtx lane_ctx(int64_t B) {
    LaneCtx x;
    x.gid = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    x.active = x.gid < B;
    x.cand = x.active ? x.gid : B - 1;
    x.wbase = static_cast<int64_t>(blockIdx.x) * kBlock + (threadIdx.x / kWave) * kWave;
    return x;
}

// Forward pass; makespan/energy outputs, the mask and the selection partials are each optional.
template <int MODE>
__global__ void __launch_bounds__(kBlock)
forward_kernel(DevGraph g, const uint8_t *__restrict__ levels, int64_t B, float *__restrict__ T_out,
               float *__restrict__ E_out, EmoTargets tg, float *cold, int64_t bpad, bool vec, int wlog) {
    extern __shared__ float4 smem4[];
    Tab<MODE> tab = make_tab<MODE>(g, smem4, wlog);
    const LaneCtx x = lane_ctx(B);
    const Row row{levels + x.cand * g.P, g.P, vec};
    f32x32 hot;
    Scratch sc{cold, nullptr, nullptr, bpad, x.gid};
    const Fwd f = run_forward<MODE, false>(g.eval, tab, g.F, g.static_power, row, hot, sc);
    if (x.active) {
        if (T_out) T_out[x.cand] = f.T;
        if (E_out) E_out[x.cand] = f.E;
    }
    if (tg.n) emo_select_all(blockIdx.x, x.active, f.T, f.E, x.cand, B, tg);
}

// Forward + backward (slack) pass with the same optional outputs.
template <int MODE, bool STAGED>
__global__ void __launch_bounds__(kBlock)
slack_kernel(DevGraph g, DevProgram pr, int32_t cols, const uint8_t *__restrict__ levels, int64_t B,
             float *__restrict__ S, float *__restrict__ T_out, float *__restrict__ E_out,
             EmoTargets tg, float *cold, float *keep, float *cold_bwd, int64_t bpad, bool vec, int wlog) {
    extern __shared__ float4 smem4[];
    Tab<MODE> tab = make_tab<MODE>(g, smem4, wlog);
    __shared__ float stg_all[STAGED ? kWavesPerBlock : 1][STAGED ? kStage * 65 : 1];
    const LaneCtx x = lane_ctx(B);
    const Row row{levels + x.cand * g.P, g.P, vec};
    f32x32 hot;
    Scratch sc{cold, keep, cold_bwd, bpad, x.gid};
    const Fwd f = run_forward<MODE, true>(pr, tab, g.F, g.static_power, row, hot, sc);
    if (x.active) {
        if (T_out) T_out[x.cand] = f.T;
        if (E_out) E_out[x.cand] = f.E;
    }
    float *stg = STAGED ? stg_all[threadIdx.x / kWave] : nullptr;
    run_backward<MODE, STAGED>(pr, tab, g.F, f.bad ? 0.f : f.T, f.bad, row, hot, sc, S, cols, x.cand,
                               x.active, stg, x.wbase, B);
    if (tg.n) emo_select_all(blockIdx.x, x.active, f.T, f.E, x.cand, B, tg);
}

// ---------------------------------------------------------------- time-interval policies

// Forward pass for a time-interval policy (the policy form of Sec. IV-A; Alg. 1): the row holds
// one level per interval [T_i, T_{i+1}) of the batch's change points (T_0 = 0, the last interval
// open-ended), a pack runs at the level of the interval that holds its start time, and the
// energy adds each interval's idle power times the wall time it covers inside [0, makespan).
// `pts` (K - 1 change points, increasing) and `idle` (F values) are in LDS.  With NREG > 0
// (K - 1 <= NREG) the change points are also held in registers `rp` (uniform values, padded with
// +infinity) and a pack's interval is the count of points <= its start, an unrolled sequence of
// compares with no memory access on the dependency chain; otherwise a binary search over LDS.
constexpr int kIvRegPoints = 15;

template <int MODE, int NREG>
__device__ __forceinline__ Fwd run_forward_iv(const DevProgram &pr, Tab<MODE> &tab, int F, const Row &row,
                                              int K, const float *pts, const float *rp, const float *idle,
                                              f32x32 &hot, const Scratch &sc) {
    u32x32 lw;
    int lgroup = -1;
    bool bad = false;   // any level byte >= F in the row (the idle term reads every interval's)
    for (int i = 0; i < K; ++i) bad |= level_at(row, lw, lgroup, i) >= static_cast<unsigned>(F);
    // the level of a lane-dependent interval: with NREG > 0 (K <= 16) from the row's four words
    // by a two-level select; otherwise a byte load from the row (indexing the register bank with
    // a lane-dependent index would cost a select per word of the bank)
    unsigned q0 = 0u, q1 = 0u, q2 = 0u, q3 = 0u;
    if (NREG > 0) {
        if (row.vec) {
            const uint4 v = *reinterpret_cast<const uint4 *>(row.row);
            q0 = v.x; q1 = v.y; q2 = v.z; q3 = v.w;
        } else {
            for (int i = 0; i < K; ++i) {
                const unsigned b = static_cast<unsigned>(row.row[i]) << ((i & 3) * 8);
                if (i < 4) q0 |= b;
                else if (i < 8) q1 |= b;
                else if (i < 12) q2 |= b;
                else q3 |= b;
            }
        }
    }
    float T = pr.t_const;
    double eacc = 0.0;
    float eblk = 0.f;
    int nblk = 0;
    const int n = pr.n_ops;
    for (int i = 0; i < n; ++i) {
        const FwdStep st = ld_prog(pr.fwd, i);
        const uint32_t flags = uni(st.flags);
        const int32_t pack = uni(st.pack);
        const int32_t nin = uni(st.in_count);
        const int32_t ib = uni(st.in_begin);
        float est = __uint_as_float(uni(st.cst));
        for (int j = 0; j < nin; ++j)
            est = fmaxf(est, slot_get(hot, sc.cold, sc.bpad, sc.col, uni(ld_prog(pr.ins, ib + j))));
        float dur;
        if (pack >= 0) {
            int lo = 0, hi = K - 1;   // number of change points <= est
            if (NREG > 0) {
#pragma unroll
                for (int j = 0; j < NREG; ++j) lo += rp[j] <= est ? 1 : 0;
            } else {
                while (lo < hi) {
                    const int mid = (lo + hi) >> 1;
                    if (pts[mid] <= est) lo = mid + 1;
                    else hi = mid;
                }
            }
            unsigned l;
            if (NREG > 0) {
                const unsigned wd = lo < 8 ? (lo < 4 ? q0 : q1) : (lo < 12 ? q2 : q3);
                l = (wd >> ((lo & 3) * 8)) & 0xffu;
            } else {
                l = row.row[lo];
            }
            l = l < static_cast<unsigned>(F) ? l : 0u;
            const float2 te = tab.get(pack, static_cast<int>(l), 1);
            dur = te.x;
            eblk += te.y;
            if (++nblk == kEnergyBlock) {
                eacc += static_cast<double>(eblk);
                eblk = 0.f;
                nblk = 0;
            }
        } else {
            dur = __uint_as_float(uni(st.dur));
        }
        const float eft = est + dur;
        if (flags & kStepOut) slot_set(hot, sc.cold, sc.bpad, sc.col, uni(st.out), eft);
        if (flags & kStepSink) T = fmaxf(T, eft);
    }
    eacc += static_cast<double>(eblk);
    // idle energy, interval by interval in increasing order: the whole length of each interval
    // that ends at or before the makespan, then the part of the next one below it
    const double Td = static_cast<double>(T);
    for (int i = 0; i < K; ++i) {
        const double lo = i > 0 ? static_cast<double>(pts[i - 1]) : 0.0;
        if (!(Td > lo)) break;   // this interval and the later ones start at or after T
        const bool whole = i < K - 1 && pts[i] <= T;
        const double d = whole ? static_cast<double>(pts[i]) - lo : Td - lo;
        unsigned l = level_at(row, lw, lgroup, i);
        l = l < static_cast<unsigned>(F) ? l : 0u;
        eacc = fma(static_cast<double>(idle[l]), d, eacc);
        if (!whole) break;
    }
    Fwd f;
    f.E = static_cast<float>(eacc);
    f.T = T;
    f.bad = bad;
    if (bad) {
        f.T = __builtin_nanf("");
        f.E = __builtin_nanf("");
    }
    return f;
}

template <int MODE, int NREG>
__global__ void __launch_bounds__(kBlock)
interval_kernel(DevGraph g, IvPolicy pol, const uint8_t *__restrict__ levels, int64_t B,
                float *__restrict__ T_out, float *__restrict__ E_out, EmoTargets tg, float *cold,
                int64_t bpad, bool vec,
                int wlog) {
    extern __shared__ float4 smem4[];
    __shared__ float s_pts[kMaxIntervals];
    __shared__ float s_idle[kMaxLevels];
    for (int i = threadIdx.x; i < pol.K - 1; i += kBlock) s_pts[i] = pol.pts[i];
    for (int i = threadIdx.x; i < g.F; i += kBlock) s_idle[i] = pol.idle[i];
    __syncthreads();
    Tab<MODE> tab = make_tab<MODE>(g, smem4, wlog);
    const LaneCtx x = lane_ctx(B);
    const Row row{levels + x.cand * pol.K, pol.K, vec};
    f32x32 hot;
    Scratch sc{cold, nullptr, nullptr, bpad, x.gid};
    float rp[NREG > 0 ? NREG : 1];
#pragma unroll
    for (int j = 0; j < NREG; ++j) rp[j] = j < pol.K - 1 ? pol.pts[j] : __builtin_inff();
    const Fwd f = run_forward_iv<MODE, NREG>(g.eval, tab, g.F, row, pol.K, s_pts, rp, s_idle, hot, sc);
    if (x.active) {
        if (T_out) T_out[x.cand] = f.T;
        if (E_out) E_out[x.cand] = f.E;
    }
    if (tg.n) emo_select_all(blockIdx.x, x.active, f.T, f.E, x.cand, B, tg);
}

// ---------------------------------------------------------------- selection (Eq. 4)

static_assert(sizeof(EmoSel) == sizeof(emo_selection), "result layout");
static_assert(sizeof(EmoPartial) == kPartialBytes, "partial record layout");

__global__ void empty_result(emo_selection *res) {
    EmoSel *r = reinterpret_cast<EmoSel *>(res);
    r->index = -1;
    r->energy = __builtin_nanf("");
    r->makespan = __builtin_nanf("");
    r->num_feasible = 0;
}

// Stage 2 of the selection: one workgroup of kFinThreads reduces the n partial records into the
// emo_selection record.  It is latency-bound, so each thread keeps four independent loads in
// flight and a round covers 4 * kFinThreads records (all of them up to 4M candidates).
constexpr int kFinThreads = 1024;
constexpr int kFinWaves = kFinThreads / kWave;

__global__ void __launch_bounds__(kFinThreads)
select_finalize_kernel(const EmoPartial *__restrict__ parts, int64_t n, emo_selection *results) {
    // workgroup k: target k's records
    const EmoPartial *__restrict__ part = parts + static_cast<int64_t>(blockIdx.x) * n;
    emo_selection *res = results + blockIdx.x;
    __shared__ unsigned long long s_key[kFinWaves];
    __shared__ float s_T[kFinWaves];
    __shared__ unsigned long long s_cnt[kFinWaves];
    unsigned long long key = ~0ull;
    float T = 0.f;
    unsigned long long cnt = 0;
    for (int64_t base = threadIdx.x; base < n; base += 4 * kFinThreads) {
        EmoPartial p[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int64_t i = base + k * kFinThreads;
            if (i < n) {
                p[k] = part[i];
            } else {
                p[k].key = ~0ull;
                p[k].count = 0;
                p[k].makespan = 0.f;
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            cnt += p[k].count;
            if (p[k].key < key) {
                key = p[k].key;
                T = p[k].makespan;
            }
        }
    }
    emo_wave_min_key(&key, &T);
    for (int off = kWave / 2; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off, kWave);
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    if (lane == 0) {
        s_key[wave] = key;
        s_T[wave] = T;
        s_cnt[wave] = cnt;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    for (int w = 1; w < kFinWaves; ++w) {
        if (s_key[w] < key) {
            key = s_key[w];
            T = s_T[w];
        }
        cnt += s_cnt[w];
    }
    EmoSel *r = reinterpret_cast<EmoSel *>(res);
    if (key == ~0ull) {
        r->index = -1;
        r->energy = __builtin_nanf("");
        r->makespan = __builtin_nanf("");
    } else {
        r->index = static_cast<int64_t>(key & 0xffffffffull);
        r->energy = __uint_as_float(static_cast<unsigned int>(key >> 32));
        r->makespan = T;
    }
    r->num_feasible = static_cast<int64_t>(cnt);
}

// Selection from stored makespans and energies: each lane takes kSelPer consecutive candidates
// (16-byte loads when both arrays are 16-byte aligned), so a workgroup covers kSelGroup
// candidates and writes one partial record for them.  A wave covers 8 mask words: the lanes
// 8j .. 8j+7 hold the 32 candidates of word j, four bits each.
constexpr int kSelPer = 4;
constexpr int64_t kSelGroup = static_cast<int64_t>(kBlock) * kSelPer;

__global__ void __launch_bounds__(kBlock)
select_results_kernel(const float *__restrict__ T, const float *__restrict__ E, int64_t B, EmoTargets tg,
                      bool vec) {
    __shared__ unsigned long long s_key[kWavesPerBlock];
    __shared__ float s_T[kWavesPerBlock];
    __shared__ unsigned int s_cnt[kWavesPerBlock];
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kSelGroup + static_cast<int64_t>(threadIdx.x) * kSelPer;
    float t[kSelPer], e[kSelPer];
    if (vec && c0 + kSelPer <= B) {
        const float4 tv = *reinterpret_cast<const float4 *>(T + c0);
        const float4 ev = *reinterpret_cast<const float4 *>(E + c0);
        t[0] = tv.x; t[1] = tv.y; t[2] = tv.z; t[3] = tv.w;
        e[0] = ev.x; e[1] = ev.y; e[2] = ev.z; e[3] = ev.w;
    } else {
#pragma unroll
        for (int k = 0; k < kSelPer; ++k) {
            const bool in = c0 + k < B;
            t[k] = in ? T[c0 + k] : 0.f;
            e[k] = in ? E[c0 + k] : 0.f;
        }
    }
    // the targets one after another from the same loaded makespans and energies
    for (int j = 0; j < tg.n; ++j) {
        const float target = tg.t[j];
        unsigned int *mask = tg.mask[j];
        EmoPartial *part = tg.part ? tg.part + j * tg.nparts : nullptr;
        unsigned int nib = 0u;
        unsigned long long key = ~0ull;
        float kT = 0.f;
#pragma unroll
        for (int k = 0; k < kSelPer; ++k) {
            const bool feas = c0 + k < B && t[k] <= target;   // false for NaN
            nib |= feas ? 1u << k : 0u;
            const unsigned long long kk = feas ? (static_cast<unsigned long long>(__float_as_uint(e[k])) << 32) |
                                                     static_cast<unsigned long long>(c0 + k)
                                               : ~0ull;
            if (kk < key) {
                key = kk;
                kT = t[k];
            }
        }
        if (mask) {
            unsigned int w = nib << (kSelPer * (lane & 7));
            w |= __shfl_xor(w, 1, kWave);
            w |= __shfl_xor(w, 2, kWave);
            w |= __shfl_xor(w, 4, kWave);
            const int64_t word = c0 / 32;
            if ((lane & 7) == 0 && word * 32 < B) mask[word] = w;
        }
        if (!part) continue;
        emo_wave_min_key(&key, &kT);
        unsigned int cnt = static_cast<unsigned int>(__popc(nib));
        for (int off = kWave / 2; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off, kWave);
        if (j > 0) __syncthreads();   // the previous target's records have been read
        if (lane == 0) {
            s_key[wave] = key;
            s_T[wave] = kT;
            s_cnt[wave] = cnt;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            EmoPartial p;
            p.key = s_key[0];
            p.makespan = s_T[0];
            p.count = s_cnt[0];
            for (int w = 1; w < kWavesPerBlock; ++w) {
                if (s_key[w] < p.key) {
                    p.key = s_key[w];
                    p.makespan = s_T[w];
                }
                p.count += s_cnt[w];
            }
            part[blockIdx.x] = p;
        }
    }
}

int64_t grid_for(int64_t B) { return (B + kBlock - 1) / kBlock; }

size_t table_bytes(const DevGraph &g) {
    return (static_cast<size_t>(g.P) * g.F + kTablePad) * sizeof(float2);
}

bool vec_levels(const DevGraph &g, const uint8_t *levels) {
    return g.P % 16 == 0 && reinterpret_cast<uintptr_t>(levels) % 16 == 0;
}

// Packs per table window (a power of two) so that one window of rows fills kWindowBytes.
int window_log(const DevGraph &g) {
    int wlog = 0;
    while ((static_cast<size_t>(2) << wlog) * g.F * sizeof(float2) <= static_cast<size_t>(kWindowBytes)) ++wlog;
    return wlog;
}

// Table mode for a launch with `other_lds` bytes of LDS already in use.
int table_mode(const DevGraph &g, const DevProgram &prog, size_t other_lds, size_t *dyn) {
    const size_t tb = table_bytes(g);
    if (tb + other_lds <= kLdsBudget) {
        *dyn = tb;
        return kTabLds;
    }
    const size_t wb = 2 * static_cast<size_t>(kWindowBytes);
    // a window holds at least two packs' rows (so its start is 16-byte aligned)
    if (prog.monotone && window_log(g) >= 1 && wb + other_lds <= kLdsBudget) {
        *dyn = wb;
        return kTabWindow;
    }
    *dyn = 0;
    return kTabGlobal;
}

}  // namespace

int64_t forward_blocks(int64_t B) { return grid_for(B); }

int64_t select_results_blocks(int64_t B) { return (B + kSelGroup - 1) / kSelGroup; }

size_t forward_scratch_bytes(const DevProgram &prog, int64_t B) {
    return static_cast<size_t>(prog.n_cold) * static_cast<size_t>(grid_for(B) * kBlock) * sizeof(float);
}

size_t slack_scratch_bytes(const DevProgram &prog, int64_t B) {
    const size_t rows = static_cast<size_t>(prog.n_cold) + static_cast<size_t>(prog.n_ops) +
                        static_cast<size_t>(prog.n_cold_bwd);
    return rows * static_cast<size_t>(grid_for(B) * kBlock) * sizeof(float);
}

static_assert(sizeof(EmoTargets) == sizeof(SelTargets) && offsetof(EmoTargets, part) == offsetof(SelTargets, part) &&
                  offsetof(EmoTargets, t) == offsetof(SelTargets, t) &&
                  offsetof(EmoTargets, mask) == offsetof(SelTargets, mask),
              "the targets' kernel argument layout");
EmoTargets dev_targets(const SelTargets &tg) {
    EmoTargets d;
    std::memcpy(&d, &tg, sizeof(d));
    return d;
}

hipError_t launch_forward(const DevGraph &g, const uint8_t *levels, int64_t B, float *T, float *E,
                          const SelTargets &tg, void *scratch, hipStream_t s) {
    const int64_t grid = grid_for(B);
    const int64_t bpad = grid * kBlock;
    float *cold = g.eval.n_cold > 0 ? static_cast<float *>(scratch) : nullptr;
    size_t dyn = 0;
    const int mode = table_mode(g, g.eval, 0, &dyn);
    const bool vec = vec_levels(g, levels);
    const int wlog = window_log(g);
    const EmoTargets dt = dev_targets(tg);
    const dim3 gd(static_cast<unsigned>(grid)), bd(kBlock);
#define EMO_FWD_ARGS g, levels, B, T, E, dt, cold, bpad, vec, wlog
    if (mode == kTabLds) hipLaunchKernelGGL(forward_kernel<kTabLds>, gd, bd, dyn, s, EMO_FWD_ARGS);
    else if (mode == kTabWindow) hipLaunchKernelGGL(forward_kernel<kTabWindow>, gd, bd, dyn, s, EMO_FWD_ARGS);
    else hipLaunchKernelGGL(forward_kernel<kTabGlobal>, gd, bd, dyn, s, EMO_FWD_ARGS);
#undef EMO_FWD_ARGS
    return hipGetLastError();
}

hipError_t launch_slack(const DevGraph &g, const DevProgram &prog, int32_t out_cols,
                        const uint8_t *levels, int64_t B, float *slack, float *T, float *E,
                        const SelTargets &tg, void *scratch, hipStream_t s) {
    const int64_t grid = grid_for(B);
    const int64_t bpad = grid * kBlock;
    const size_t n_cold = static_cast<size_t>(prog.n_cold), n_keep = static_cast<size_t>(prog.n_ops),
                 n_cold_b = static_cast<size_t>(prog.n_cold_bwd);
    const size_t total = (n_cold + n_keep + n_cold_b) * static_cast<size_t>(bpad);
    float *buf = total > 0 ? static_cast<float *>(scratch) : nullptr;
    float *cold = buf;
    float *keep = buf ? buf + n_cold * bpad : nullptr;
    float *cold_b = buf ? keep + n_keep * bpad : nullptr;
    // staged output needs packs visited in increasing id and whole 32-pack segments
    const bool staged = out_cols == g.P && prog.monotone && g.P % kStage == 0 &&
                        reinterpret_cast<uintptr_t>(slack) % 16 == 0;
    const size_t stage_bytes = staged ? static_cast<size_t>(kWavesPerBlock) * kStage * 65 * sizeof(float) : 0;
    size_t dyn = 0;
    const int mode = table_mode(g, prog, stage_bytes, &dyn);
    const bool vec = vec_levels(g, levels);
    const int wlog = window_log(g);
    const EmoTargets dt = dev_targets(tg);
    const dim3 gd(static_cast<unsigned>(grid)), bd(kBlock);
#define EMO_SLACK_ARGS g, prog, out_cols, levels, B, slack, T, E, dt, cold, keep, cold_b, bpad, vec, wlog
    if (mode == kTabLds && staged) hipLaunchKernelGGL((slack_kernel<kTabLds, true>), gd, bd, dyn, s, EMO_SLACK_ARGS);
    else if (mode == kTabLds) hipLaunchKernelGGL((slack_kernel<kTabLds, false>), gd, bd, dyn, s, EMO_SLACK_ARGS);
    else if (mode == kTabWindow && staged) hipLaunchKernelGGL((slack_kernel<kTabWindow, true>), gd, bd, dyn, s, EMO_SLACK_ARGS);
    else if (mode == kTabWindow) hipLaunchKernelGGL((slack_kernel<kTabWindow, false>), gd, bd, dyn, s, EMO_SLACK_ARGS);
    else if (staged) hipLaunchKernelGGL((slack_kernel<kTabGlobal, true>), gd, bd, dyn, s, EMO_SLACK_ARGS);
    else hipLaunchKernelGGL((slack_kernel<kTabGlobal, false>), gd, bd, dyn, s, EMO_SLACK_ARGS);
#undef EMO_SLACK_ARGS
    return hipGetLastError();
}

hipError_t launch_intervals(const DevGraph &g, const IvPolicy &pol, const uint8_t *levels, int64_t B,
                            float *T, float *E, const SelTargets &tg, void *scratch, hipStream_t s) {
    const int64_t grid = grid_for(B);
    const int64_t bpad = grid * kBlock;
    float *cold = g.eval.n_cold > 0 ? static_cast<float *>(scratch) : nullptr;
    size_t dyn = 0;
    const int mode = table_mode(g, g.eval, 0, &dyn);
    const bool vec = pol.K % 16 == 0 && reinterpret_cast<uintptr_t>(levels) % 16 == 0;
    const int wlog = window_log(g);
    const EmoTargets dt = dev_targets(tg);
    const dim3 gd(static_cast<unsigned>(grid)), bd(kBlock);
#define EMO_IV_ARGS g, pol, levels, B, T, E, dt, cold, bpad, vec, wlog
    const bool reg = pol.K - 1 <= kIvRegPoints;
    if (mode == kTabLds && reg) hipLaunchKernelGGL((interval_kernel<kTabLds, kIvRegPoints>), gd, bd, dyn, s, EMO_IV_ARGS);
    else if (mode == kTabLds) hipLaunchKernelGGL((interval_kernel<kTabLds, 0>), gd, bd, dyn, s, EMO_IV_ARGS);
    else if (mode == kTabWindow && reg) hipLaunchKernelGGL((interval_kernel<kTabWindow, kIvRegPoints>), gd, bd, dyn, s, EMO_IV_ARGS);
    else if (mode == kTabWindow) hipLaunchKernelGGL((interval_kernel<kTabWindow, 0>), gd, bd, dyn, s, EMO_IV_ARGS);
    else if (reg) hipLaunchKernelGGL((interval_kernel<kTabGlobal, kIvRegPoints>), gd, bd, dyn, s, EMO_IV_ARGS);
    else hipLaunchKernelGGL((interval_kernel<kTabGlobal, 0>), gd, bd, dyn, s, EMO_IV_ARGS);
#undef EMO_IV_ARGS
    return hipGetLastError();
}

hipError_t launch_empty_result(emo_selection *res, hipStream_t s) {
    hipLaunchKernelGGL(empty_result, dim3(1), dim3(1), 0, s, res);
    return hipGetLastError();
}

hipError_t launch_select_finalize(const SelTargets &tg, emo_selection *results, hipStream_t s) {
    if (tg.n < 1 || !tg.part) return hipSuccess;
    hipLaunchKernelGGL(select_finalize_kernel, dim3(static_cast<unsigned>(tg.n)), dim3(kFinThreads), 0, s,
                       static_cast<const EmoPartial *>(tg.part), tg.nparts, results);
    return hipGetLastError();
}

hipError_t launch_select_results(const float *T, const float *E, int64_t B, const SelTargets &tg,
                                 hipStream_t s) {
    if (tg.n < 1) return hipSuccess;
    const bool vec = (reinterpret_cast<uintptr_t>(T) | reinterpret_cast<uintptr_t>(E)) % 16 == 0;
    hipLaunchKernelGGL(select_results_kernel, dim3(static_cast<unsigned>(select_results_blocks(B))), dim3(kBlock),
                       0, s, T, E, B, dev_targets(tg), vec);
    return hipGetLastError();
}

int64_t noalloc_max_candidates() {
    return static_cast<int64_t>(kNoAllocScratchBytes / kPartialBytes) * kSelGroup;
}

hipError_t noalloc_scratch(int dev, void **out) {
    static std::mutex mu;
    static void *addr[kNoAllocMaxDevices] = {};
    if (dev < 0 || dev >= kNoAllocMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        // the caller has made `dev` current: this is that device's copy of the array
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

}  // namespace emo
