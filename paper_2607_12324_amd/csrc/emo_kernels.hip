// HIP kernels for gfx950: batched what-if evaluation of per-pack frequency policies.
//
// Layout: one candidate policy per lane.  Every lane of a wave walks the same compiled program
// (the graph is shared by all candidates), so the program, its predecessor lists and the table
// base offsets are wave-uniform and come through scalar loads; only the level bytes, the table
// entries they select and the finish times differ per lane.
//
// Per step (one node in topological order, Eq. 1 and Alg. 1):
//   EST = max(cst, finish times of candidate-dependent predecessors)
//   EFT = EST + dur,  dur = table time at the pack's level (Eq. 3) or the fixed duration
// The makespan is the running max (Eq. 2); pack energies are summed in fp32 blocks of 64 packs
// that are added into an fp64 total, and the static term static_power * T closes Eq. 2.
//
// Finish-time slots live in LDS (slot k of lane L at [k][L] in the wave's region, conflict
// free) when they fit, otherwise in device scratch laid out [slot][candidate] so that a wave's
// access to one slot is one contiguous 256-byte segment.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "emo_internal.h"
#include "emo_select.h"

namespace emo {
namespace {

constexpr int kBlock = EMO_BLOCK;
constexpr int kWave = EMO_WAVE;
constexpr int kWavesPerBlock = EMO_WAVES_PER_BLOCK;
constexpr int kEnergyBlock = 64;
constexpr size_t kLdsBudget = 60 * 1024;   // dynamic LDS, leaves room for static LDS under 64 KB

struct Slots {
    float *lds;        // this wave's LDS region, or nullptr
    float *glob;       // device scratch [slot][Bpad], or nullptr
    int64_t stride;    // Bpad
    int64_t col;       // this lane's column in the scratch
    int lane;
    __device__ __forceinline__ float &at(int k) const {
        return lds ? lds[k * kWave + lane] : glob[static_cast<int64_t>(k) * stride + col];
    }
};

struct Fwd {
    float T;
    float E;
    bool bad;
};

__device__ __forceinline__ float2 table_at(const float2 *tab_lds, const float2 *tab, int idx) {
    return tab_lds ? tab_lds[idx] : tab[idx];
}

// Forward pass of one candidate (row = its level bytes).
__device__ Fwd forward(const DevProgram &pr, const float2 *tab_lds, const float2 *tab, int F,
                       float static_power, const uint8_t *row, const Slots &sl) {
    float T = pr.t_const;
    double eacc = 0.0;
    float eblk = 0.f;
    int nblk = 0;
    bool bad = false;
    for (int i = 0; i < pr.n_ops; ++i) {
        const Op op = pr.op[i];
        const int2 r = pr.in_range[i];
        float est = __uint_as_float(op.cst);
        for (int j = r.x; j < r.y; ++j) est = fmaxf(est, sl.at(pr.ins[j]));
        float dur;
        if (op.pack >= 0) {
            unsigned l = row[op.pack];
            bad |= (l >= static_cast<unsigned>(F));
            l = l < static_cast<unsigned>(F) ? l : 0u;
            const float2 te = table_at(tab_lds, tab, op.pack * F + static_cast<int>(l));
            dur = te.x;
            eblk += te.y;
            if (++nblk == kEnergyBlock) {
                eacc += static_cast<double>(eblk);
                eblk = 0.f;
                nblk = 0;
            }
        } else {
            dur = __uint_as_float(op.dur);
        }
        const float eft = est + dur;
        if (op.out >= 0) sl.at(op.out) = eft;
        T = fmaxf(T, eft);
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

// Stage the (time, energy) table into LDS when it fits.
__device__ const float2 *stage_table(const DevGraph &g, float2 *smem_tab, bool use_lds) {
    if (!use_lds) return nullptr;
    const int n = g.P * g.F;
    for (int i = threadIdx.x; i < n; i += blockDim.x) smem_tab[i] = g.tab[i];
    __syncthreads();
    return smem_tab;
}

struct LaunchShape {
    bool tab_lds;
    bool slot_lds;
    size_t tab_bytes;
    size_t slot_bytes;   // per block
    size_t lds_bytes;
};

LaunchShape shape_for(const DevGraph &g, int n_slots) {
    LaunchShape s;
    s.tab_bytes = static_cast<size_t>(g.P) * g.F * sizeof(float2);
    s.tab_lds = s.tab_bytes <= 32 * 1024;
    size_t tb = s.tab_lds ? (s.tab_bytes + 15) / 16 * 16 : 0;
    size_t sb = static_cast<size_t>(n_slots) * kWave * sizeof(float) * kWavesPerBlock;
    s.slot_lds = tb + sb <= kLdsBudget;
    s.slot_bytes = s.slot_lds ? sb : 0;
    s.lds_bytes = tb + s.slot_bytes;
    return s;
}

struct Ctx {
    const float2 *tab_lds;
    Slots sl;
    int64_t c;        // candidate of this lane (clamped to B-1 for idle lanes)
    bool active;
};

__device__ Ctx make_ctx(const DevGraph &g, int n_slots, bool tab_lds, bool slot_lds,
                        float *gslots, int64_t bpad, int64_t B) {
    extern __shared__ float4 smem4[];
    char *smem = reinterpret_cast<char *>(smem4);
    const size_t tab_bytes = static_cast<size_t>(g.P) * g.F * sizeof(float2);
    const size_t tb = tab_lds ? (tab_bytes + 15) / 16 * 16 : 0;
    Ctx x;
    x.tab_lds = stage_table(g, reinterpret_cast<float2 *>(smem), tab_lds);
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    x.active = gid < B;
    x.c = x.active ? gid : B - 1;
    x.sl.lane = lane;
    x.sl.col = gid;
    x.sl.stride = bpad;
    x.sl.lds = slot_lds ? reinterpret_cast<float *>(smem + tb) + static_cast<size_t>(wave) * n_slots * kWave : nullptr;
    x.sl.glob = slot_lds ? nullptr : gslots;
    return x;
}

// Forward pass; makespan/energy outputs, the mask and the selection partials are each optional.
__global__ void __launch_bounds__(kBlock)
forward_kernel(DevGraph g, const uint8_t *__restrict__ levels, int64_t B, float *__restrict__ T_out,
               float *__restrict__ E_out, float target, uint32_t *__restrict__ mask,
               EmoPartial *part, bool tab_lds, bool slot_lds, float *gslots, int64_t bpad) {
    Ctx x = make_ctx(g, g.eval.n_slots, tab_lds, slot_lds, gslots, bpad, B);
    Fwd f = forward(g.eval, x.tab_lds, g.tab, g.F, g.static_power, levels + x.c * g.P, x.sl);
    if (x.active) {
        if (T_out) T_out[x.c] = f.T;
        if (E_out) E_out[x.c] = f.E;
    }
    if (mask || part) emo_select_block(x.active, f.T, f.E, x.c, B, target, mask, part);
}

__global__ void __launch_bounds__(kBlock)
slack_kernel(DevGraph g, DevProgram pr, int32_t cols, const uint8_t *__restrict__ levels, int64_t B,
             float *__restrict__ slack, float *__restrict__ T_out, float *__restrict__ E_out,
             float target, uint32_t *__restrict__ mask, EmoPartial *part,
             bool tab_lds, bool slot_lds, float *gslots, int64_t bpad) {
    Ctx x = make_ctx(g, pr.n_slots, tab_lds, slot_lds, gslots, bpad, B);
    const uint8_t *row = levels + x.c * g.P;
    Fwd f = forward(pr, x.tab_lds, g.tab, g.F, g.static_power, row, x.sl);
    if (x.active) {
        if (T_out) T_out[x.c] = f.T;
        if (E_out) E_out[x.c] = f.E;
    }
    // backward: slot i holds EFT of step i, replaced by its latest start time LST
    const float T = f.T;
    const float inf = __builtin_inff();
    float *out_row = slack + x.c * static_cast<int64_t>(cols);
    for (int i = pr.n_ops - 1; i >= 0; --i) {
        const Op op = pr.op[i];
        const int2 sr = pr.succ_range[i];
        float lft = T;
        if (sr.y > sr.x) {
            lft = inf;
            for (int j = sr.x; j < sr.y; ++j) lft = fminf(lft, x.sl.at(pr.succs[j]));
        }
        float dur;
        if (op.pack >= 0) {
            unsigned l = row[op.pack];
            l = l < static_cast<unsigned>(g.F) ? l : 0u;
            dur = table_at(x.tab_lds, g.tab, op.pack * g.F + static_cast<int>(l)).x;
        } else {
            dur = __uint_as_float(op.dur);
        }
        const float eft = x.sl.at(i);
        x.sl.at(i) = lft - dur;
        const int col = pr.out_col[i];
        if (x.active && col >= 0) out_row[col] = f.bad ? __builtin_nanf("") : lft - eft;
    }
    if (mask || part) emo_select_block(x.active, f.T, f.E, x.c, B, target, mask, part);
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

__global__ void __launch_bounds__(kBlock)
select_finalize_kernel(const EmoPartial *__restrict__ part, int64_t n, emo_selection *res) {
    emo_select_finalize(part, n, res);
}

__global__ void __launch_bounds__(kBlock)
select_results_kernel(const float *__restrict__ T, const float *__restrict__ E, int64_t B,
                      float target, uint32_t *__restrict__ mask, EmoPartial *part) {
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const bool active = gid < B;
    const int64_t c = active ? gid : B - 1;
    emo_select_block(active, T[c], E[c], c, B, target, mask, part);
}

int64_t grid_for(int64_t B) { return (B + kBlock - 1) / kBlock; }

// Device scratch for finish-time slots that do not fit in LDS.
hipError_t scratch(size_t bytes, hipStream_t s, float **p) {
    *p = nullptr;
    if (bytes == 0) return hipSuccess;
    return hipMallocAsync(reinterpret_cast<void **>(p), bytes, s);
}

}  // namespace

hipError_t launch_forward(const DevGraph &g, const uint8_t *levels, int64_t B, float *T, float *E,
                          float target, uint32_t *mask, void *part, hipStream_t s) {
    LaunchShape sh = shape_for(g, g.eval.n_slots);
    const int64_t grid = grid_for(B);
    const int64_t bpad = grid * kBlock;
    float *gs = nullptr;
    hipError_t e = scratch(sh.slot_lds ? 0 : static_cast<size_t>(g.eval.n_slots) * bpad * 4, s, &gs);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(forward_kernel, dim3(static_cast<unsigned>(grid)), dim3(kBlock), sh.lds_bytes, s,
                       g, levels, B, T, E, target, mask, static_cast<EmoPartial *>(part), sh.tab_lds,
                       sh.slot_lds, gs, bpad);
    e = hipGetLastError();
    if (gs) {
        hipError_t e2 = hipFreeAsync(gs, s);
        if (e == hipSuccess) e = e2;
    }
    return e;
}

hipError_t launch_slack(const DevGraph &g, const DevProgram &prog, int32_t out_cols,
                        const uint8_t *levels, int64_t B, float *slack, float *T, float *E,
                        float target, uint32_t *mask, void *part, hipStream_t s) {
    LaunchShape sh = shape_for(g, prog.n_slots);
    const int64_t grid = grid_for(B);
    const int64_t bpad = grid * kBlock;
    float *gs = nullptr;
    hipError_t e = scratch(sh.slot_lds ? 0 : static_cast<size_t>(prog.n_slots) * bpad * 4, s, &gs);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(slack_kernel, dim3(static_cast<unsigned>(grid)), dim3(kBlock), sh.lds_bytes, s,
                       g, prog, out_cols, levels, B, slack, T, E, target, mask,
                       static_cast<EmoPartial *>(part), sh.tab_lds, sh.slot_lds, gs, bpad);
    e = hipGetLastError();
    if (gs) {
        hipError_t e2 = hipFreeAsync(gs, s);
        if (e == hipSuccess) e = e2;
    }
    return e;
}

int64_t forward_blocks(int64_t B) { return grid_for(B); }

hipError_t launch_empty_result(emo_selection *res, hipStream_t s) {
    hipLaunchKernelGGL(empty_result, dim3(1), dim3(1), 0, s, res);
    return hipGetLastError();
}

hipError_t launch_select_finalize(const void *part, int64_t nparts, emo_selection *res,
                                  hipStream_t s) {
    hipLaunchKernelGGL(select_finalize_kernel, dim3(1), dim3(kBlock), 0, s,
                       static_cast<const EmoPartial *>(part), nparts, res);
    return hipGetLastError();
}

hipError_t launch_select_results(const float *T, const float *E, int64_t B, float target,
                                 uint32_t *mask, void *part, hipStream_t s) {
    hipLaunchKernelGGL(select_results_kernel, dim3(static_cast<unsigned>(grid_for(B))), dim3(kBlock), 0, s,
                       T, E, B, target, mask, static_cast<EmoPartial *>(part));
    return hipGetLastError();
}

}  // namespace emo
