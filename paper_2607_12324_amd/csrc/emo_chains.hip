// Chain-lane kernels for graphs whose candidate-dependent part is a set of disjoint chains —
// for example kernels in stream order whose other predecessors are candidate-independent host
// launch nodes (folded into constant start-time floors).  Such a graph has little parallelism
// per candidate along a chain but one independent chain per stream, so each candidate gets
// `lanes` lanes (a power of two at least the number of chains, at most 64), one per chain.
//
// Per step of a chain (Eq. 1 and Alg. 1 with at most one candidate-dependent predecessor):
//   EFT = max(EFT of the previous step, cst) + dur
// where cst is the latest finish among the step's candidate-independent predecessors and dur the
// pack's table time at its level (Eq. 3) or the node's fixed duration.  The makespan is the max
// over the chains' last finish times and the candidate-independent makespan (Eq. 2).  Padding
// steps (cst = 0, dur = 0, no pack) leave a chain's finish time unchanged, since finish times
// are >= 0.  Pack energies are summed per chain in fp32 blocks of 64 steps added into fp64, and
// the chains' sums are added in fp64 across the candidate's lanes; this order differs from the
// program order of the other kernel kinds, so energies agree with them to the same 1e-5 bound
// but not bit for bit.  Makespans and slack use the same fp32 operations and are identical.
//
// Slack (backward pass, total float): each chain walks its steps in reverse; a step's latest
// finish is the latest start of the next step on its chain (T after the chain's last step), and
// slack = latest finish - EFT.  Finish times are not stored: the forward pass checkpoints the
// finish time entering each block of kStepBlock steps, and the backward pass recomputes a block's
// finish times from its checkpoint (4 bytes per 16 steps of scratch instead of 4 per step).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "emo_internal.h"

namespace emo {
namespace {

constexpr int kChainBlockThreads = 1024;
constexpr int K = kChainStepBlock;
constexpr int kEnergySteps = 64;   // fp32 energy block (steps of one chain)
constexpr int kStageBytes = 32 * 1024;

// Plain variant (the rows of a block do not fit the LDS stage): every lane reads its own table
// entries from device memory.
template <bool SLACK>
__global__ void __launch_bounds__(kChainBlockThreads)
chains_kernel(DevGraph g, DevChains c, const uint8_t *__restrict__ levels, int64_t B,
              float *__restrict__ To, float *__restrict__ Eo, float *__restrict__ S,
              float *__restrict__ ck, int64_t pitch) {
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kChainBlockThreads + threadIdx.x;
    const int64_t cand0 = gid >> c.lane_log;
    const int j = static_cast<int>(threadIdx.x) & (c.lanes - 1);
    const bool active = cand0 < B;
    const int64_t cand = active ? cand0 : B - 1;
    const uint8_t *__restrict__ row = levels + cand * g.P;
    const ChainStep *__restrict__ st = c.steps + j;
    const int F = g.F;
    const unsigned Fu = static_cast<unsigned>(F);
    const int nblk = c.len / K;
    float f = 0.f, eb = 0.f;
    double ed = 0.0;
    unsigned bad = 0u;
    for (int b = 0; b < nblk; ++b) {
        if (SLACK) ck[static_cast<int64_t>(b) * pitch + gid] = f;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const ChainStep r = st[static_cast<int64_t>(b * K + i) << c.lane_log];
            const unsigned lv = r.pack >= 0 ? row[r.pack] : 0u;
            bad |= lv >= Fu ? 1u : 0u;
            const unsigned l = lv < Fu ? lv : 0u;
            const float2 te = r.pack >= 0 ? g.tab[static_cast<int64_t>(r.pack) * F + l] : make_float2(r.dur, 0.f);
            f = fmaxf(f, r.cst) + te.x;
            eb += te.y;
        }
        if ((b + 1) % (kEnergySteps / K) == 0) {
            ed += static_cast<double>(eb);
            eb = 0.f;
        }
    }
    ed += static_cast<double>(eb);
    float T = f;
    for (int off = 1; off < c.lanes; off <<= 1) {
        T = fmaxf(T, __shfl_xor(T, off));
        ed += __shfl_xor(ed, off);
        bad |= __shfl_xor(bad, off);
    }
    T = fmaxf(T, c.t_const);
    float E = static_cast<float>(ed + static_cast<double>(g.static_power) * static_cast<double>(T));
    if (bad) {
        T = __builtin_nanf("");
        E = __builtin_nanf("");
    }
    if (active && j == 0) {
        To[cand] = T;
        Eo[cand] = E;
    }
    if (!SLACK) return;
    const float nan = __builtin_nanf("");
    float lft = bad ? 0.f : T;
    for (int b = nblk - 1; b >= 0; --b) {
        float fb = ck[static_cast<int64_t>(b) * pitch + gid];
        int pk[K];
        float ti[K], fi[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const ChainStep r = st[static_cast<int64_t>(b * K + i) << c.lane_log];
            pk[i] = r.pack;
            const unsigned lv = r.pack >= 0 ? row[r.pack] : 0u;
            const unsigned l = lv < Fu ? lv : 0u;
            ti[i] = r.pack >= 0 ? g.tabt[static_cast<int64_t>(r.pack) * F + l] : r.dur;
            fb = fmaxf(fb, r.cst) + ti[i];
            fi[i] = fb;
        }
#pragma unroll
        for (int i = K - 1; i >= 0; --i) {
            if (active && pk[i] >= 0) S[cand * g.P + pk[i]] = bad ? nan : lft - fi[i];
            lft = lft - ti[i];
        }
    }
}

// Staged variant (a block's table rows fit kStageBytes): at step k every candidate of the
// workgroup visits the same packs, so the workgroup copies the rows of a block's K x lanes packs
// into LDS once (about 16x less L2 traffic than every lane reading its entry out of a different
// row), and the loop is software-pipelined so that no memory round trip is exposed:
//   - step records of block b+2 are copied into a 3-deep LDS ring,
//   - table rows of block b+1 are copied into the other half of a double buffer,
//   - level bytes of block b+1 are loaded into registers,
// all while block b is computed from LDS and registers; one barrier per block.  The backward
// pass runs the same pipeline downwards (blocks b-2, b-1), reading times only.
// LDS: rows [2][K * lanes * F] (float2 forward, float backward) | records [3][K * lanes].
constexpr int kRowsPerThread = kStageBytes / 8 / kChainBlockThreads;   // float2 entries

// S here is the chain-ordered slack scratch [B][len * lanes] (row pitch srow); a second kernel
// (gather_slack) writes it out in pack order.
template <bool SLACK>
__global__ void __launch_bounds__(kChainBlockThreads)
chains_staged(DevGraph g, DevChains c, const uint8_t *__restrict__ levels, int64_t B,
              float *__restrict__ To, float *__restrict__ Eo, float *__restrict__ S,
              float *__restrict__ ck, int64_t pitch) {
    const int64_t srow = static_cast<int64_t>(c.len) << c.lane_log;
    extern __shared__ float4 smem[];
    const int t = threadIdx.x;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kChainBlockThreads + t;
    const int64_t cand0 = gid >> c.lane_log;
    const int j = t & (c.lanes - 1);
    const bool active = cand0 < B;
    const int64_t cand = active ? cand0 : B - 1;
    const uint8_t *__restrict__ row = levels + cand * g.P;
    const int F = g.F;
    const int nslot = K * c.lanes;
    const int nrow = nslot * F;
    const int nblk = c.len / K;
    float2 *rows2 = reinterpret_cast<float2 *>(smem);                 // forward: [2][nrow]
    float *rows1 = reinterpret_cast<float *>(smem);                   // backward: [2][nrow]
    ChainStep *recs = reinterpret_cast<ChainStep *>(rows2 + 2 * nrow); // [3][nslot]
    const ChainStep *__restrict__ gsteps = c.steps;
    auto rec_slot = [&](int b) { return recs + (b % 3) * nslot; };
    const unsigned Fu = static_cast<unsigned>(F);

    // ------------------------------------------------------------------ forward
    if (t < nslot) rec_slot(0)[t] = gsteps[t];
    if (nblk > 1 && t < nslot) rec_slot(1)[t] = gsteps[nslot + t];
    __syncthreads();
    for (int q = 0; q < kRowsPerThread; ++q) {
        const int e = t + q * kChainBlockThreads;
        if (e < nrow) {
            const int32_t pk = rec_slot(0)[e / F].pack;
            rows2[e] = pk >= 0 ? g.tab[static_cast<int64_t>(pk) * F + e % F] : make_float2(0.f, 0.f);
        }
    }
    unsigned lcur[K];
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const int32_t pk = rec_slot(0)[(i << c.lane_log) + j].pack;
        lcur[i] = pk >= 0 ? row[pk] : 0u;
    }
    __syncthreads();
    float f = 0.f, eb = 0.f;
    double ed = 0.0;
    unsigned bad = 0u;
    for (int b = 0; b < nblk; ++b) {
        if (SLACK) ck[static_cast<int64_t>(b) * pitch + gid] = f;
        const bool more = b + 1 < nblk;
        // prefetch: records of block b+2, rows and level bytes of block b+1
        ChainStep rpre{-1, 0.f, 0.f, 0};
        if (b + 2 < nblk && t < nslot) rpre = gsteps[static_cast<int64_t>(b + 2) * nslot + t];
        float2 rowpre[kRowsPerThread];
        unsigned lnext[K];
        if (more) {
            const ChainStep *rn = rec_slot(b + 1);
#pragma unroll
            for (int q = 0; q < kRowsPerThread; ++q) {
                const int e = t + q * kChainBlockThreads;
                const int32_t pk = e < nrow ? rn[e / F].pack : -1;
                rowpre[q] = pk >= 0 ? g.tab[static_cast<int64_t>(pk) * F + e % F] : make_float2(0.f, 0.f);
            }
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const int32_t pk = rn[(i << c.lane_log) + j].pack;
                lnext[i] = pk >= 0 ? row[pk] : 0u;
            }
        }
        // block b from LDS and registers
        const ChainStep *rb = rec_slot(b);
        const float2 *rowb = rows2 + (b & 1) * nrow;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const int slot = (i << c.lane_log) + j;
            const ChainStep r = rb[slot];
            bad |= lcur[i] >= Fu ? 1u : 0u;
            const unsigned l = lcur[i] < Fu ? lcur[i] : 0u;
            const float2 tv = rowb[slot * F + l];
            const float2 te = r.pack >= 0 ? tv : make_float2(r.dur, 0.f);
            f = fmaxf(f, r.cst) + te.x;
            eb += te.y;
        }
        if ((b + 1) % (kEnergySteps / K) == 0) {
            ed += static_cast<double>(eb);
            eb = 0.f;
        }
        // commit the prefetched block: its buffers were last read before the previous barrier
        if (more) {
            float2 *dst = rows2 + ((b + 1) & 1) * nrow;
#pragma unroll
            for (int q = 0; q < kRowsPerThread; ++q) {
                const int e = t + q * kChainBlockThreads;
                if (e < nrow) dst[e] = rowpre[q];
            }
        }
        if (b + 2 < nblk && t < nslot) rec_slot(b + 2)[t] = rpre;
        __syncthreads();
        if (more) {
#pragma unroll
            for (int i = 0; i < K; ++i) lcur[i] = lnext[i];
        }
    }
    ed += static_cast<double>(eb);
    float T = f;
    for (int off = 1; off < c.lanes; off <<= 1) {
        T = fmaxf(T, __shfl_xor(T, off));
        ed += __shfl_xor(ed, off);
        bad |= __shfl_xor(bad, off);
    }
    T = fmaxf(T, c.t_const);
    float E = static_cast<float>(ed + static_cast<double>(g.static_power) * static_cast<double>(T));
    if (bad) {
        T = __builtin_nanf("");
        E = __builtin_nanf("");
    }
    if (active && j == 0) {
        To[cand] = T;
        Eo[cand] = E;
    }
    if (!SLACK) return;

    // ------------------------------------------------------------------ backward
    const float nan = __builtin_nanf("");
    float lft = bad ? 0.f : T;
    const int top = nblk - 1;
    __syncthreads();   // the forward pass is done with every buffer
    if (t < nslot) rec_slot(top)[t] = gsteps[static_cast<int64_t>(top) * nslot + t];
    if (top >= 1 && t < nslot) rec_slot(top - 1)[t] = gsteps[static_cast<int64_t>(top - 1) * nslot + t];
    __syncthreads();
    for (int q = 0; q < 2 * kRowsPerThread; ++q) {
        const int e = t + q * kChainBlockThreads;
        if (e < nrow) {
            const int32_t pk = rec_slot(top)[e / F].pack;
            rows1[(top & 1) * nrow + e] = pk >= 0 ? g.tabt[static_cast<int64_t>(pk) * F + e % F] : 0.f;
        }
    }
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const int32_t pk = rec_slot(top)[(i << c.lane_log) + j].pack;
        lcur[i] = pk >= 0 ? row[pk] : 0u;
    }
    float fb = ck[static_cast<int64_t>(top) * pitch + gid];
    __syncthreads();
    for (int b = top; b >= 0; --b) {
        const bool more = b >= 1;
        ChainStep rpre{-1, 0.f, 0.f, 0};
        if (b >= 2 && t < nslot) rpre = gsteps[static_cast<int64_t>(b - 2) * nslot + t];
        float rowpre[2 * kRowsPerThread];
        unsigned lnext[K];
        float fnext = 0.f;
        if (more) {
            const ChainStep *rn = rec_slot(b - 1);
#pragma unroll
            for (int q = 0; q < 2 * kRowsPerThread; ++q) {
                const int e = t + q * kChainBlockThreads;
                const int32_t pk = e < nrow ? rn[e / F].pack : -1;
                rowpre[q] = pk >= 0 ? g.tabt[static_cast<int64_t>(pk) * F + e % F] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const int32_t pk = rn[(i << c.lane_log) + j].pack;
                lnext[i] = pk >= 0 ? row[pk] : 0u;
            }
            fnext = ck[static_cast<int64_t>(b - 1) * pitch + gid];
        }
        const ChainStep *rb = rec_slot(b);
        const float *rowb = rows1 + (b & 1) * nrow;
        float ti[K], fi[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const int slot = (i << c.lane_log) + j;
            const ChainStep r = rb[slot];
            const unsigned l = lcur[i] < Fu ? lcur[i] : 0u;
            ti[i] = r.pack >= 0 ? rowb[slot * F + l] : r.dur;
            fb = fmaxf(fb, r.cst) + ti[i];
            fi[i] = fb;
        }
        // slack in chain order: the candidate's lanes write 4 * lanes contiguous bytes per step
        float *__restrict__ so = S + cand * srow + (static_cast<int64_t>(b) * K << c.lane_log) + j;
#pragma unroll
        for (int i = K - 1; i >= 0; --i) {
            so[i << c.lane_log] = bad ? nan : lft - fi[i];
            lft = lft - ti[i];
        }
        if (more) {
            float *dst = rows1 + ((b - 1) & 1) * nrow;
#pragma unroll
            for (int q = 0; q < 2 * kRowsPerThread; ++q) {
                const int e = t + q * kChainBlockThreads;
                if (e < nrow) dst[e] = rowpre[q];
            }
        }
        if (b >= 2 && t < nslot) rec_slot(b - 2)[t] = rpre;
        __syncthreads();
        if (more) {
#pragma unroll
            for (int i = 0; i < K; ++i) lcur[i] = lnext[i];
            fb = fnext;
        }
    }
}

// Pack-order slack rows from the chain-ordered scratch: thread (c, q) writes packs 4q..4q+3 of
// candidate c (one 16-byte store; 64 lanes cover 1 KB of a row) from their chain positions,
// which are nearly in order (packs are launched round-robin-like over the streams).
constexpr int kGatherThreads = 256;
__global__ void __launch_bounds__(kGatherThreads)
gather_slack(const float *__restrict__ tmp, const int32_t *__restrict__ pos, int64_t B, int32_t P,
             int64_t srow, float *__restrict__ S) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kGatherThreads + threadIdx.x;
    const int64_t per_row = P / 4;
    const int64_t cand = q / per_row;
    if (cand >= B) return;
    const int32_t p = static_cast<int32_t>(q - cand * per_row) * 4;
    const float *__restrict__ src = tmp + cand * srow;
    float4 v;
    v.x = src[pos[p]];
    v.y = src[pos[p + 1]];
    v.z = src[pos[p + 2]];
    v.w = src[pos[p + 3]];
    *reinterpret_cast<float4 *>(S + cand * P + p) = v;
}

int64_t chain_grid(const DevChains &c, int64_t B) {
    return ((B << c.lane_log) + kChainBlockThreads - 1) / kChainBlockThreads;
}

}  // namespace

namespace {
// Whether the staged kernel applies, and whether slack goes through the chain-ordered scratch
// (staged kernel, P a multiple of 4).
bool staged_ok(const DevGraph &g, const DevChains &c) {
    return static_cast<size_t>(K) * c.lanes * g.F * sizeof(float2) <= static_cast<size_t>(kStageBytes);
}
size_t round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
}  // namespace

size_t chains_scratch_bytes(const DevGraph &g, const DevChains &c, int64_t B, bool slack) {
    const size_t lanes = static_cast<size_t>(chain_grid(c, B)) * kChainBlockThreads;
    const size_t ck = slack ? round256(static_cast<size_t>(c.len / K) * lanes * sizeof(float)) : 0;
    const size_t tmp = slack && staged_ok(g, c) && g.P % 4 == 0
                           ? round256(static_cast<size_t>(B) * (static_cast<size_t>(c.len) << c.lane_log) * sizeof(float))
                           : 0;
    return ck + tmp + 2 * round256(static_cast<size_t>(B) * sizeof(float));
}

hipError_t launch_chains(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                         float *T, float *E, float *slack, float target, uint32_t *mask, void *part,
                         void *scratch, hipStream_t s) {
    const int64_t grid = chain_grid(c, B);
    const int64_t pitch = grid * kChainBlockThreads;
    const bool st = staged_ok(g, c);
    const bool via_tmp = slack && st && g.P % 4 == 0;
    char *p = static_cast<char *>(scratch);
    float *ck = slack ? reinterpret_cast<float *>(p) : nullptr;
    if (slack) p += round256(static_cast<size_t>(c.len / K) * pitch * sizeof(float));
    const int64_t srow = static_cast<int64_t>(c.len) << c.lane_log;
    float *tmp = via_tmp ? reinterpret_cast<float *>(p) : nullptr;
    if (via_tmp) p += round256(static_cast<size_t>(B) * srow * sizeof(float));
    const size_t vec = round256(static_cast<size_t>(B) * sizeof(float));
    float *Ts = T ? T : reinterpret_cast<float *>(p);
    float *Es = E ? E : reinterpret_cast<float *>(p + vec);
    const dim3 gd(static_cast<unsigned>(grid)), bd(kChainBlockThreads);
    const size_t nslot = static_cast<size_t>(K) * c.lanes;
    const size_t dyn = st ? 2 * nslot * g.F * sizeof(float2) + 3 * nslot * sizeof(ChainStep) : 0;
    if (via_tmp) hipLaunchKernelGGL((chains_staged<true>), gd, bd, dyn, s, g, c, levels, B, Ts, Es, tmp, ck, pitch);
    else if (slack) hipLaunchKernelGGL((chains_kernel<true>), gd, bd, 0, s, g, c, levels, B, Ts, Es, slack, ck, pitch);
    else if (st) hipLaunchKernelGGL((chains_staged<false>), gd, bd, dyn, s, g, c, levels, B, Ts, Es, slack, ck, pitch);
    else hipLaunchKernelGGL((chains_kernel<false>), gd, bd, 0, s, g, c, levels, B, Ts, Es, slack, ck, pitch);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && via_tmp) {
        const int64_t n = B * (g.P / 4);
        hipLaunchKernelGGL(gather_slack, dim3(static_cast<unsigned>((n + kGatherThreads - 1) / kGatherThreads)),
                           dim3(kGatherThreads), 0, s, tmp, c.pos, B, g.P, srow, slack);
        e = hipGetLastError();
    }
    if (e == hipSuccess && (mask || part)) e = launch_select_results(Ts, Es, B, target, mask, part, s);
    return e;
}

}  // namespace emo
