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

#include <atomic>

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

// ---------------------------------------------------------------- windowed variant
//
// The lane-per-chain kernels above read each candidate's level bytes at the packs its chains
// are at; when the chains drift thousands of pack ids apart (streams launched in random order),
// every 8-step block of a wave touches up to 64 different cache lines, and slack has to be
// written in chain order and gathered.  The windowed kernel cuts the pack ids into windows of
// W packs instead and turns the layout around: a wave is 64 candidates on ONE chain, and a
// workgroup is G groups of 64 candidates x nc chains.  Per window the workgroup copies into
// LDS, with 16-byte loads issued two windows ahead into registers:
//   - the G*64 candidates' level bytes of the window (checked against F on the way),
//   - the window's table rows (time and energy; times only in the second pass),
//   - the window's step block: where each chain's steps start, and the step records.
// Each wave then walks its chain's steps inside the window (the count varies per chain; waves
// meet at the window's barrier).  Slack comes from a second pass over the windows (below), which
// writes each step's slack into an LDS tile [candidate][column] that the workgroup writes out in
// pack order with 16-byte stores.
//
// Column W of every level row is 0 and row W of the table is zero, so a fixed node (column W)
// reads a zero time and energy and adds its own duration; its tile entry is column W's pad.
// Energies are summed per chain in fp32 over each window, added into fp64, and the chains'
// sums are added in chain order.
constexpr int kWinPre = 4;                         // 16-byte prefetch pieces per thread and window
constexpr size_t kWinLds = 150 * 1024;
constexpr size_t kWinSpare = 1024;                   // chains_scan_full: 16 spare bytes per lane
constexpr int kWinMaxWaves = 16;

__host__ __device__ inline uint32_t round16u(uint32_t x) { return (x + 15u) & ~15u; }

struct WinLayout {
    uint32_t lvl_pitch;    // bytes per candidate row of a level buffer (W + 4)
    uint32_t lvl_buf;      // bytes of one level buffer
    uint32_t off_bad;      // u32 [NC]: candidate has a level >= F
    uint32_t off_tfin;     // f32 [NC]: makespan (NaN when bad)
    uint32_t off_blk;      // [2] step blocks
    uint32_t off_x;        // phase region: tables (forward, backward), chain sums, slack tile
    uint32_t tab_elems;    // entries of one table buffer ((W + 1) * F)
    uint32_t off_tile;     // f32 [NC][W + 1] (backward)
    uint32_t total;
};

__host__ __device__ inline WinLayout win_layout(int W, int NC, int F, int nwaves, int blk_bytes) {
    WinLayout L;
    L.lvl_pitch = static_cast<uint32_t>(W) + 4u;
    L.lvl_buf = round16u(static_cast<uint32_t>(NC) * L.lvl_pitch);
    L.off_bad = 2u * L.lvl_buf;
    L.off_tfin = L.off_bad + 4u * static_cast<uint32_t>(NC);
    L.off_blk = round16u(L.off_tfin + 4u * static_cast<uint32_t>(NC));
    L.off_x = L.off_blk + 2u * static_cast<uint32_t>(blk_bytes);
    // entries per table buffer, a multiple of 4 so that the second buffer starts 16-byte
    // aligned for its 16-byte stores (with fp32 or float2 entries)
    L.tab_elems = (static_cast<uint32_t>(W + 1) * static_cast<uint32_t>(F) + 3u) & ~3u;
    // (256 spare float2 entries: a lookup with an invalid level byte reads at most 255 entries
    // past a table buffer; the backward tables are followed by the slack tile)
    const uint32_t fwd = (2u * L.tab_elems + 256u) * 8u;
    const uint32_t comb = 64u * 8u * kWinMaxWaves + static_cast<uint32_t>(nwaves) * 64u * 4u;
    L.off_tile = L.off_x + round16u(2u * L.tab_elems * 4u);
    const uint32_t bwd = L.off_tile - L.off_x + static_cast<uint32_t>(NC) * static_cast<uint32_t>(W + 1) * 4u;
    uint32_t m = fwd > comb ? fwd : comb;
    m = m > bwd ? m : bwd;
    L.total = L.off_x + m;
    return L;
}

__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Bit 7 of every byte of a word that holds a level >= F (F <= 128: a byte b < 128 gets bit 7
// from (b + 128 - F) exactly when b >= F, and a byte >= 128 has it already).
__device__ __forceinline__ uint32_t bad_levels(uint32_t x, uint32_t addf) {
    return (((x & 0x7f7f7f7fu) + addf) | x) & 0x80808080u;
}

// max of two non-negative finite floats: their bit patterns order like unsigned integers, and
// the integer max needs none of the NaN-quieting that the compiler adds to fmaxf on operands
// loaded from memory.  Finish times and start floors here are always >= 0 and finite.
__device__ __forceinline__ float fmax_nonneg(float a, float b) {
    const unsigned x = __float_as_uint(a), y = __float_as_uint(b);
    return __uint_as_float(x > y ? x : y);
}


struct WinArgs {
    int W, wlog, nc, NC, F;
    int blk_bytes, hdr_words;
    int slots_lvl, slots_tab8, slots_tab4, slots_blk;   // prefetch slots per category
    WinLayout L;
};

// Prefetch slots of each category for nt threads; false when they exceed kWinPre.
__host__ __device__ inline bool win_slots(int W, int NC, int F, int blk_bytes, int nt, int *sl, int *st8,
                                          int *st4, int *sb) {
    *sl = (NC * (W / 16) + nt - 1) / nt;
    *st8 = (W * F / 2 + nt - 1) / nt;
    *st4 = (W * F / 4 + nt - 1) / nt;
    *sb = (blk_bytes / 16 + nt - 1) / nt;
    return *sl + *st8 + *sb <= kWinPre;
}

// One window's copy in flight: the thread's pieces (16 bytes each), slot by slot: the first
// slots hold level rows, the next table rows, the next the step block (how many of each is the
// same for every thread, so the category of a slot is uniform); which of them read as zero
// (level columns past P, table rows past the last pack, pieces past the end).  Rows of a pack
// count that is not a multiple of 16 are not 16-byte aligned (the layout then gives every
// thread one level piece, in slot 0): the piece is the five dwords around it (v[0] and x, from
// its address rounded down to 4 bytes), and meta holds its byte shift (2 bits) and its number
// of bytes before the row's end (5 bits).
struct WinSet {
    uint4 v[kWinPre];
    uint32_t x;
    uint32_t zero;
    uint32_t meta;
};

// Issues exactly kWinPre loads for window w (a piece past the end reads a valid address and is
// zeroed when stored; unused slots read the first block piece), with the addresses as scalar
// bases plus 32-bit lane offsets, so that the compiler counts them and waits at a commit for
// the older window's loads only.  esize: bytes per table entry (8 forward, 4 backward).
template <bool ROWS16>
__device__ __forceinline__ void win_load(const WinArgs &a, const uint8_t *__restrict__ levels,
                                         const void *__restrict__ tab, int esize,
                                         const uint4 *__restrict__ blocks, int64_t base, int64_t B,
                                         int32_t P, int w, WinSet &s) {
    const int t = threadIdx.x, nt = blockDim.x;
    const int rlog = a.wlog - 4;                                   // pieces per level row: W / 16
    const int n_lvl = a.NC << rlog;
    const int n_tab = (a.W * a.F * esize) >> 4;
    const int n_blk = a.blk_bytes >> 4;
    const int s_lvl = a.slots_lvl, s_tab = esize == 8 ? a.slots_tab8 : a.slots_tab4;
    const int64_t wcol = static_cast<int64_t>(w) << a.wlog;
    const uint8_t *lbase = levels + base * P + wcol;               // window's first column, row base
    const int64_t tab_off = wcol * a.F * esize;                    // bytes
    const uint32_t tab_left = static_cast<uint32_t>(static_cast<int64_t>(P) * a.F * esize - tab_off);
    const char *tbase = static_cast<const char *>(tab) + tab_off;
    const char *bbase = reinterpret_cast<const char *>(blocks + static_cast<int64_t>(w) * n_blk);
    const int64_t rows_left = B - base;                             // rows of this workgroup in range
    const int64_t cols_left = P - wcol;
    uint32_t zero = 0u, meta = 0u;
#pragma unroll
    for (int i = 0; i < kWinPre; ++i) {
        const char *src;
        uint32_t off;
        bool z;
        if (i < s_lvl) {
            const int q = t + i * nt;
            const int r = q >> rlog, k = q - (r << rlog);
            const int rr = r < rows_left ? r : static_cast<int>(rows_left - 1);
            z = q >= n_lvl || 16 * k >= cols_left;
            off = z ? 0u : static_cast<uint32_t>(rr) * static_cast<uint32_t>(P) + 16u * static_cast<uint32_t>(k);
            src = reinterpret_cast<const char *>(lbase);
            if (!ROWS16 && i == 0) {
                // the five dwords from the piece's address rounded down to 4 bytes; a dword at or
                // past the last one of the batch's rows reads that last dword instead (its bytes
                // are all past the row's end, and masked when stored)
                const uint64_t at = reinterpret_cast<uint64_t>(src + off);
                const uint64_t lo = reinterpret_cast<uint64_t>(levels);
                const uint64_t last = (lo + static_cast<uint64_t>(B * P) + 3u) / 4u * 4u - 4u;
                const uint64_t al = at & ~static_cast<uint64_t>(3);
                uint32_t d[5];
#pragma unroll
                for (int j = 0; j < 5; ++j) {
                    const uint64_t aj = al + 4u * j;
                    d[j] = *reinterpret_cast<const uint32_t *>(aj <= last ? aj : last);
                }
                s.v[0] = make_uint4(d[0], d[1], d[2], d[3]);
                s.x = d[4];
                const int64_t nb = cols_left - 16 * k;
                meta = static_cast<uint32_t>(at & 3u) | (static_cast<uint32_t>(nb < 16 ? (nb > 0 ? nb : 0) : 16) << 2);
                zero |= z ? 1u << i : 0u;
                continue;
            }
        } else if (i < s_lvl + s_tab) {
            const int q = t + (i - s_lvl) * nt;
            z = q >= n_tab || 16u * static_cast<uint32_t>(q) >= tab_left;
            off = z ? 0u : 16u * static_cast<uint32_t>(q);
            src = tbase;
        } else {
            const int q = t + (i - s_lvl - s_tab) * nt;
            z = q >= n_blk || i >= s_lvl + s_tab + a.slots_blk;
            off = z ? 0u : 16u * static_cast<uint32_t>(q);
            src = bbase;
        }
        zero |= z ? 1u << i : 0u;
        s.v[i] = *reinterpret_cast<const uint4 *>(src + off);
    }
    s.zero = zero;
    s.meta = meta;
}

// A level piece of an unaligned row from its five dwords: the 16 bytes at the piece's shift,
// with the bytes past the row's end cleared.
__device__ __forceinline__ uint4 win_piece(const WinSet &s) {
    const uint32_t sh = s.meta & 3u, nb = (s.meta >> 2) & 31u;
    uint32_t o[4];
    o[0] = __builtin_amdgcn_alignbyte(s.v[0].y, s.v[0].x, sh);
    o[1] = __builtin_amdgcn_alignbyte(s.v[0].z, s.v[0].y, sh);
    o[2] = __builtin_amdgcn_alignbyte(s.v[0].w, s.v[0].z, sh);
    o[3] = __builtin_amdgcn_alignbyte(s.x, s.v[0].w, sh);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t keep = nb >= 4u * j + 4u ? 4u : (nb > 4u * j ? nb - 4u * j : 0u);   // bytes kept
        o[j] &= keep == 4u ? 0xffffffffu : (1u << (8u * keep)) - 1u;
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// Copies window w's pieces into LDS buffer `buf`; a level byte >= F marks its candidate in `bad`
// when it is given (the forward pass).  Such a byte is not cleared: the candidate's makespan,
// energy and slack become NaN whatever its lookups read, and a lookup at column c <= W with
// level l <= 255 stays inside the workgroup's LDS (at most 255 entries past the window's table,
// which the layout leaves room for).
template <bool ROWS16>
__device__ __forceinline__ void win_store(const WinArgs &a, char *lds, int buf, void *tabbuf, int esize,
                                          uint32_t *bad, uint32_t addf, const WinSet &s) {
    const int t = threadIdx.x, nt = blockDim.x;
    const int rlog = a.wlog - 4;
    const int n_lvl = a.NC << rlog;
    const int n_tab = (a.W * a.F * esize) >> 4;
    const int n_blk = a.blk_bytes >> 4;
    const int s_lvl = a.slots_lvl, s_tab = esize == 8 ? a.slots_tab8 : a.slots_tab4;
    uint8_t *lvl = reinterpret_cast<uint8_t *>(lds) + buf * a.L.lvl_buf;
    uint4 *blk = reinterpret_cast<uint4 *>(lds + a.L.off_blk + buf * a.blk_bytes);
#pragma unroll
    for (int i = 0; i < kWinPre; ++i) {
        uint4 v = !ROWS16 && i == 0 ? win_piece(s) : s.v[i];
        if ((s.zero >> i) & 1u) v = make_uint4(0u, 0u, 0u, 0u);
        if (i < s_lvl) {
            const int q = t + i * nt;
            if (q < n_lvl) {
                const int r = q >> rlog, k = q - (r << rlog);
                uint32_t *d = reinterpret_cast<uint32_t *>(lvl + r * a.L.lvl_pitch + 16 * k);
                d[0] = v.x;
                d[1] = v.y;
                d[2] = v.z;
                d[3] = v.w;
                if (bad && (bad_levels(v.x, addf) | bad_levels(v.y, addf) | bad_levels(v.z, addf) |
                            bad_levels(v.w, addf)))
                    bad[r] = 1u;
            }
        } else if (i < s_lvl + s_tab) {
            const int q = t + (i - s_lvl) * nt;
            if (q < n_tab) reinterpret_cast<uint4 *>(tabbuf)[q] = v;
        } else if (i < s_lvl + s_tab + a.slots_blk) {
            const int q = t + (i - s_lvl - s_tab) * nt;
            if (q < n_blk) blk[q] = v;
        }
    }
}

// Buffer resources of the planned copies: raw buffer accesses with a 32-bit per-lane offset and a
// uniform offset, and the hardware's range check (an access at or past `bytes` reads zeros and
// writes nothing).  The fourth word is the CDNA3/CDNA4 raw-buffer configuration.
typedef unsigned int emo_u4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t win_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}
// An offset past every planned buffer (they all hold less than 2^31 bytes, and a uniform offset
// stays below 2^31 too): loads there read zeros and stores are dropped.
constexpr uint32_t kWinNoStore = 0x80000000u;

// The copy of a window wholly inside the graph (its W columns and table rows all exist), with
// each thread's pieces at offsets fixed for the whole kernel: win_plan computes them once, and a
// window then costs its loads, its stores and a few scalar operations.  A thread with no piece
// in a slot loads past the slot's buffer (the range check returns zeros without touching memory)
// and stores them to its lane's spare 16 bytes at LDS offset `spare` (so every load is waited
// for and every store made on every path, which keeps the compiler's count of loads in flight
// exact).
struct WinPlan {
    uint32_t src[kWinPre];    // byte offset of the piece in its slot's per-window source
    uint32_t dst0[kWinPre];   // LDS byte offset of the piece in buffer 0 (or the spare)
    uint32_t dst1[kWinPre];   // in buffer 1
    uint32_t has;             // bit i: the thread has a piece in slot i
};

template <int NT>
__device__ __forceinline__ WinPlan win_plan(const WinArgs &a, int esize, int64_t rows_left, int32_t P,
                                            uint32_t spare) {
    const int t = threadIdx.x, nt = blockDim.x;
    const int rlog = a.wlog - 4;
    const int n_lvl = a.NC << rlog;
    const int n_tab = (a.W * a.F * esize) >> 4;
    const int n_blk = a.blk_bytes >> 4;
    const int s_lvl = 1, s_tab = NT;
    const uint32_t own = spare + 16u * static_cast<uint32_t>(t & 63);
    WinPlan p;
    p.has = 0u;
#pragma unroll
    for (int i = 0; i < kWinPre; ++i) {
        bool ok = false;
        uint32_t src = 0u, d0 = 0u, stride = 0u;
        if (i < s_lvl) {
            const int q = t + i * nt;
            const int r = q >> rlog, k = q - (r << rlog);
            const int rr = r < rows_left ? r : static_cast<int>(rows_left - 1);
            ok = q < n_lvl;
            src = static_cast<uint32_t>(rr) * static_cast<uint32_t>(P) + 16u * static_cast<uint32_t>(k);
            d0 = static_cast<uint32_t>(r) * a.L.lvl_pitch + 16u * static_cast<uint32_t>(k);
            stride = a.L.lvl_buf;
        } else if (i < s_lvl + s_tab) {
            const int q = t + (i - s_lvl) * nt;
            ok = q < n_tab;
            src = 16u * static_cast<uint32_t>(q);
            d0 = a.L.off_x + 16u * static_cast<uint32_t>(q);
            stride = a.L.tab_elems * static_cast<uint32_t>(esize);
        } else if (i == s_lvl + s_tab) {
            const int q = t + (i - s_lvl - s_tab) * nt;
            ok = q < n_blk;
            src = 16u * static_cast<uint32_t>(q);
            d0 = a.L.off_blk + 16u * static_cast<uint32_t>(q);
            stride = static_cast<uint32_t>(a.blk_bytes);
        }
        // an absent piece reads past its buffer's end (zeros, with no memory traffic)
        p.src[i] = ok ? src : kWinNoStore;
        p.dst0[i] = ok ? d0 : own;   // (slots past those in use: ok is false, the spare slot)
        p.dst1[i] = ok ? d0 + stride : own;
        p.has |= ok ? 1u << i : 0u;
    }
    return p;
}

// The per-workgroup buffers of a pass's planned copies: the workgroup's level rows, the pass's
// table (8-byte entries forward, 4-byte in the second pass) and the step blocks.
struct WinBufs {
    __amdgpu_buffer_rsrc_t lvl, tab, blk;
    int32_t tab_win;   // table bytes per window: W * F * esize
};

// Issues the loads of window w (wholly inside the graph) from the plan.  The slots are fixed at
// compile time: slot 0 levels, slots 1 .. NT the table, slot NT + 1 the step block.
template <int NT>
__device__ __forceinline__ void win_load_full(const WinArgs &a, const WinPlan &p, const WinBufs &b, int w,
                                              WinSet &s) {
    // the window offsets are uniform; readfirstlane says so to the compiler (an offset it takes
    // for divergent becomes a loop over the distinct values around each load)
    const int so_lvl = __builtin_amdgcn_readfirstlane(w << a.wlog);
    const int so_tab = __builtin_amdgcn_readfirstlane(w * b.tab_win);
    const int so_blk = __builtin_amdgcn_readfirstlane(w * a.blk_bytes);
#pragma unroll
    for (int i = 0; i < NT + 2; ++i) {
        emo_u4 v;
        if (i == 0) v = __builtin_amdgcn_raw_buffer_load_b128(b.lvl, p.src[i], so_lvl, 0);
        else if (i <= NT) v = __builtin_amdgcn_raw_buffer_load_b128(b.tab, p.src[i], so_tab, 0);
        else v = __builtin_amdgcn_raw_buffer_load_b128(b.blk, p.src[i], so_blk, 0);
        s.v[i] = make_uint4(v.x, v.y, v.z, v.w);
    }
    s.zero = 0u;
}

// Stores a window loaded by win_load_full<NT> at the plan's destinations `dst` (its dst0 or
// dst1), with no branches.  In the forward pass (`badbits` given) the thread's level piece with
// a byte >= F sets bit 0 of *badbits; the caller marks the rows at the end of the pass.  hib: the
// bits of a byte at or above F when F is a power of two (then one mask test), else 0.
template <int NT>
__device__ __forceinline__ void win_store_full(const WinPlan &p, const uint32_t *dst, char *lds,
                                               uint32_t *badbits, uint32_t addf, uint32_t hib, const WinSet &s) {
#pragma unroll
    for (int i = 0; i < NT + 2; ++i) {
        const uint4 v = s.v[i];
        if (i == 0) {
            if (badbits) {
                const uint32_t b = hib ? (v.x | v.y | v.z | v.w) & hib
                                       : bad_levels(v.x, addf) | bad_levels(v.y, addf) | bad_levels(v.z, addf) |
                                             bad_levels(v.w, addf);
                *badbits |= b && (p.has & 1u) ? 1u : 0u;
            }
            // level rows are 4-byte aligned (odd pitch in words)
            uint32_t *d = reinterpret_cast<uint32_t *>(lds + dst[0]);
            d[0] = v.x;
            d[1] = v.y;
            d[2] = v.z;
            d[3] = v.w;
        } else {
            *reinterpret_cast<uint4 *>(lds + dst[i]) = v;
        }
    }
}

// Marks the rows of the forward pass's level pieces that held a byte >= F (after the pass; the
// caller's barrier then makes bad[] complete).
__device__ __forceinline__ void win_mark_bad(const WinArgs &a, uint32_t badbits, uint32_t *bad) {
    const int t = threadIdx.x, nt = blockDim.x;
    const int rlog = a.wlog - 4;
    (void)nt;
    if (badbits & 1u) bad[t >> rlog] = 1u;
}

// The slack tile's flush when every window lies wholly inside the graph, with each thread's (at
// most four) pieces at LDS and global offsets fixed for the whole kernel: piece j of the thread
// is float4 piece q = t + j * nt of the tile in the order of the general flush.  Global offsets
// are bytes from the workgroup's first row at the window's first column (32-bit: NC * P * 4 <
// 2^32).
struct FlushPlan {
    uint32_t src[4];   // LDS byte offset of the piece's first float
    uint32_t dst[4];   // byte offset in the slack rows
    uint32_t has;      // bit j: the piece exists and its row is in the batch
    uint32_t nan;      // bit j: the piece's candidate has an invalid level (its slack row is NaN)
};

// (after the forward pass: tfin holds the makespans, NaN for a candidate with an invalid level)
__device__ __forceinline__ FlushPlan flush_plan(const WinArgs &a, int64_t rows_left, int32_t P, const float *tfin) {
    const int t = threadIdx.x, nt = blockDim.x;
    const int W = a.W, prlog = a.wlog - 2;
    const int n = a.NC << prlog;
    FlushPlan f;
    f.has = 0u;
    f.nan = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int q = t + j * nt;
        int r, kk;
        if (prlog >= 4) {
            const int jj = q & 63, blk = q >> 6, kblog = prlog - 4;
            const int rg = blk >> kblog, kb = blk & ((1 << kblog) - 1);
            r = rg * 4 + (jj >> 4);
            kk = kb * 16 + (jj & 15);
        } else {
            r = q >> prlog;
            kk = q & ((1 << prlog) - 1);
        }
        const bool ok = q < n && r < rows_left;
        f.src[j] = ok ? a.L.off_tile + 4u * static_cast<uint32_t>(r * (W + 1) + 4 * kk) : a.L.off_tile;
        f.dst[j] = ok ? 4u * (static_cast<uint32_t>(r) * static_cast<uint32_t>(P) + 4u * static_cast<uint32_t>(kk))
                      : kWinNoStore;
        f.has |= ok ? 1u << j : 0u;
        const float tr = tfin[ok ? r : 0];
        f.nan |= ok && tr != tr ? 1u << j : 0u;
    }
    return f;
}

// `rows`: the workgroup's slack rows (S from its first row, a range check at the batch's end);
// pieces a thread does not have and rows past the batch store at kWinNoStore, which the range
// check drops, so no store needs a lane mask
__device__ __forceinline__ void flush_full(const FlushPlan &f, __amdgpu_buffer_rsrc_t rows, const char *lds, int w,
                                           int wlog) {
    const int so = (w << wlog) * 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float *src = reinterpret_cast<const float *>(lds + f.src[j]);
        float4 v = make_float4(src[0], src[1], src[2], src[3]);
        if ((f.nan >> j) & 1u) v = make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                                               __builtin_nanf(""));
        const emo_u4 u = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)};
        __builtin_amdgcn_raw_buffer_store_b128(u, rows, f.dst[j], so, 0);
    }
}

// The wave's step range [k0, k1) in the window's block (scalars).
__device__ __forceinline__ void win_range(const WinArgs &a, const char *lds, int buf, int ch, int &k0, int &k1) {
    const int32_t *hdr = reinterpret_cast<const int32_t *>(lds + a.L.off_blk + buf * a.blk_bytes);
    k0 = __builtin_amdgcn_readfirstlane(hdr[ch]);
    k1 = __builtin_amdgcn_readfirstlane(hdr[ch + 1]);
}

// Keeps the LDS reads issued before it from being moved down to their first use (the compiler
// would otherwise sink the next groups' reads and serialise the round trips again).
__device__ __forceinline__ void win_issue_point() { asm volatile("" ::: "memory"); }

// Four consecutive steps of the wave's chain: their records (column and table offset, start
// floor, fixed duration) and, once read, the candidate's level bytes at their columns.  A chain's
// steps in a window come in whole groups (padded with no-op steps), and every block has 8 no-op
// steps on both sides, so reading up to two groups beyond a chain's range stays in the block.
template <bool FIXED>
struct WinGroup {
    uint32_t ct[4];
    float cst[4];
    float dur[4];
    unsigned lv[4];
    __device__ __forceinline__ void read(const ChainWinStep *rs, int k) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint2 v = *reinterpret_cast<const uint2 *>(rs + k + i);
            ct[i] = v.x;
            cst[i] = __uint_as_float(v.y);
            if (FIXED) dur[i] = rs[k + i].dur;
        }
    }
    __device__ __forceinline__ void levels(const uint8_t *lrow) {
#pragma unroll
        for (int i = 0; i < 4; ++i) lv[i] = lrow[ct[i] & 0xffffu];
    }
};

// Slack (the two-pass scan) comes from a second forward pass instead of a backward one.  Along
// a chain with durations
// d_j and start floors cst_j, a step's only successor is the next step, so its latest finish is
// the makespan minus the durations after it; with Pre_i = d_1 + ... + d_i and Tot = Pre_n,
//   slack_i = LFT_i - EFT_i = (T - Tot) - (EFT_i - Pre_i),
// and D_i = EFT_i - Pre_i obeys D_i = max(D_{i-1}, cst_i - Pre_{i-1}), D_0 = 0, because
// EFT_i = max(EFT_{i-1}, cst_i) + d_i.  The forward pass also sums Tot per chain; the second pass
// walks the windows again, sums Pre in the same order, carries D and writes K - D (K = T - Tot)
// through the slack tile.  No finish time is checkpointed or recomputed backwards.  Pre stays
// below the chain's total time, so off the exact-sum grid its rounding is that of sums of that
// size, and every other value takes one rounding: slack agrees with the backward recurrence to
// rounding, and bit for bit when every time sum is exact (every time a multiple of one power of
// two u and every path below 2^24 u, so every sum and difference is exact in fp32 in any order).
template <bool SLACK, bool FIXED, bool ROWS16>
__global__ void __launch_bounds__(kChainBlockThreads)
chains_windowed(DevGraph g, DevChains c, WinArgs a, const uint4 *__restrict__ blocks,
                const uint8_t *__restrict__ levels, int64_t B, float *__restrict__ To,
                float *__restrict__ Eo, float *__restrict__ S) {
    extern __shared__ float4 smem[];
    char *lds = reinterpret_cast<char *>(smem);
    const int t = threadIdx.x, nt = blockDim.x;
    const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
    const int grp = wv / a.nc, ch = wv - grp * a.nc;
    const int lane = t & 63;
    const int cl = grp * 64 + lane;                               // candidate within the workgroup
    const int64_t base = static_cast<int64_t>(blockIdx.x) * a.NC;
    const int64_t gc = base + cl;                                 // the candidate
    const int W = a.W, F = a.F, nc = a.nc, nwin = c.nwin;
    const int32_t P = g.P;
    const WinLayout &L = a.L;
    uint8_t *lvl0 = reinterpret_cast<uint8_t *>(lds);             // [2][NC][W + 4] bytes
    uint32_t *bad = reinterpret_cast<uint32_t *>(lds + L.off_bad);
    float *tfin = reinterpret_cast<float *>(lds + L.off_tfin);
    float2 *tab2 = reinterpret_cast<float2 *>(lds + L.off_x);     // forward: [2][W + 1][F]
    float *tabt = reinterpret_cast<float *>(lds + L.off_x);       // backward: [2][W + 1][F]
    float *tile = reinterpret_cast<float *>(lds + L.off_tile);    // backward: [NC][W + 1]
    const uint32_t addf = (0x80u - static_cast<uint32_t>(F)) * 0x01010101u;
    auto recs = [&](int buf) {
        return reinterpret_cast<const ChainWinStep *>(lds + L.off_blk + buf * a.blk_bytes + 4 * a.hdr_words);
    };

    // ------------------------------------------------------------------ forward
    for (int i = t; i < a.NC; i += nt) {
        bad[i] = 0u;
        *reinterpret_cast<uint32_t *>(lvl0 + i * L.lvl_pitch + W) = 0u;
        *reinterpret_cast<uint32_t *>(lvl0 + L.lvl_buf + i * L.lvl_pitch + W) = 0u;
    }
    for (int i = t; i < F; i += nt) {
        tab2[W * F + i] = make_float2(0.f, 0.f);
        tab2[L.tab_elems + W * F + i] = make_float2(0.f, 0.f);
    }
    WinSet s0, s1;
    win_load<ROWS16>(a, levels, g.tab, 8, blocks, base, B, P, 0, s0);
    win_load<ROWS16>(a, levels, g.tab, 8, blocks, base, B, P, nwin > 1 ? 1 : 0, s1);
    lds_barrier();
    win_store<ROWS16>(a, lds, 0, tab2, 8, bad, addf, s0);
    lds_barrier();
    float f = 0.f, pre = 0.f;
    double ed = 0.0;
    // window w from buffer w & 1; `ld` takes window w + 2, `cm` holds window w + 1
    auto forward_window = [&](int w, WinSet &ld, WinSet &cm) {
        const int buf = w & 1;
        win_load<ROWS16>(a, levels, g.tab, 8, blocks, base, B, P, w + 2 < nwin ? w + 2 : nwin - 1, ld);
        const uint8_t *lrow = lvl0 + buf * L.lvl_buf + cl * L.lvl_pitch;
        const char *tb = reinterpret_cast<const char *>(tab2 + buf * L.tab_elems);
        const ChainWinStep *rs = recs(buf);
        int k0, k1;
        win_range(a, lds, buf, ch, k0, k1);
        float eb = 0.f;
        const int ng = (k1 - k0) >> 2;
        // group g of 4 steps: its table entries are read while the next group's level bytes and
        // the records of the group after it are in flight
        auto stage = [&](WinGroup<FIXED> &A, WinGroup<FIXED> &Bn, WinGroup<FIXED> &C, int g) {
            float2 te[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                te[i] = *reinterpret_cast<const float2 *>(tb + (((A.ct[i] >> 16) + A.lv[i]) << 3));
            Bn.levels(lrow);
            C.read(rs, k0 + 4 * (g + 2));
            win_issue_point();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f = fmax_nonneg(f, A.cst[i]) + te[i].x;
                if (FIXED) f += A.dur[i];
                eb += te[i].y;
                if (SLACK) {
                    pre += te[i].x;
                    if (FIXED) pre += A.dur[i];
                }
            }
        };
        WinGroup<FIXED> G0, G1, G2;
        G0.read(rs, k0);
        G1.read(rs, k0 + 4);
        G0.levels(lrow);
        // fp32 energy blocks of at most 60 steps (15 groups, a whole number of rotations)
        for (int c0 = 0; c0 < ng; c0 += 15) {
            const int c1 = ng < c0 + 15 ? ng : c0 + 15;
            for (int g = c0; g < c1; g += 3) {
                stage(G0, G1, G2, g);
                if (g + 1 >= c1) break;
                stage(G1, G2, G0, g + 1);
                if (g + 2 >= c1) break;
                stage(G2, G0, G1, g + 2);
            }
            ed += static_cast<double>(eb);
            eb = 0.f;
        }
        if (w + 1 < nwin) win_store<ROWS16>(a, lds, buf ^ 1, tab2 + (buf ^ 1) * L.tab_elems, 8, bad, addf, cm);
        lds_barrier();
    };
    for (int w = 0; w < nwin; w += 2) {
        forward_window(w, s0, s1);
        if (w + 1 < nwin) forward_window(w + 1, s1, s0);
    }
    // chains' makespans and energies -> the candidate's (chain order)
    double *esum = reinterpret_cast<double *>(lds + L.off_x);
    float *tsum = reinterpret_cast<float *>(lds + L.off_x + 8 * 64 * kWinMaxWaves);
    esum[wv * 64 + lane] = ed;
    tsum[wv * 64 + lane] = f;
    lds_barrier();
    if (ch == 0) {
        float T = c.t_const;
        double e = 0.0;
        for (int j = 0; j < nc; ++j) {
            T = fmaxf(T, tsum[(grp * nc + j) * 64 + lane]);
            e += esum[(grp * nc + j) * 64 + lane];
        }
        float E = static_cast<float>(e + static_cast<double>(g.static_power) * static_cast<double>(T));
        if (bad[cl]) {
            T = __builtin_nanf("");
            E = __builtin_nanf("");
        }
        tfin[cl] = T;
        if (gc < B) {
            To[gc] = T;
            Eo[gc] = E;
        }
    }
    if (!SLACK) return;
    lds_barrier();

    const int prlog = a.wlog - 2;                           // float4 pieces per tile row: W / 4
    // slack tile of window w -> pack order; a wave covers 4 candidates x 16 pieces when rows
    // are long enough (conflict-free LDS reads with the odd row pitch), else whole rows
    // (W is a power of two: shifts, no divisions)
    auto flush_tile = [&](int w) {
        if (!ROWS16 && (P & 3) != 0) {
            // rows of a pack count that is not a multiple of 4 (4-byte aligned only): one float
            // per lane, consecutive lanes on consecutive columns of a row (256-byte pieces)
            const int n1 = a.NC << a.wlog;
            for (int q = t; q < n1; q += nt) {
                const int r = q >> a.wlog, cc = q & (W - 1);
                const int64_t row = base + r;
                const int64_t col = (static_cast<int64_t>(w) << a.wlog) + cc;
                const float v = tfin[r] != tfin[r] ? __builtin_nanf("") : tile[r * (W + 1) + cc];
                if (row < B && col < P) S[row * P + col] = v;
            }
            return;
        }
        const int n = a.NC << prlog;
        for (int q = t; q < n; q += nt) {
            int r, kk;
            if (prlog >= 4) {
                const int j = q & 63, blk = q >> 6, kblog = prlog - 4;
                const int rg = blk >> kblog, kb = blk & ((1 << kblog) - 1);
                r = rg * 4 + (j >> 4);
                kk = kb * 16 + (j & 15);
            } else {
                r = q >> prlog;
                kk = q & ((1 << prlog) - 1);
            }
            const float *src = tile + r * (W + 1) + 4 * kk;
            float4 v = make_float4(src[0], src[1], src[2], src[3]);
            if (tfin[r] != tfin[r]) v = make_float4(__builtin_nanf(""), __builtin_nanf(""),
                                                   __builtin_nanf(""), __builtin_nanf(""));
            const int64_t row = base + r;
            const int64_t col = (static_cast<int64_t>(w) << a.wlog) + 4 * kk;
            if (row < B && col < P) *reinterpret_cast<float4 *>(S + row * P + col) = v;   // 16-byte aligned
        }
    };
    for (int i = t; i < F; i += nt) {
        tabt[W * F + i] = 0.f;
        tabt[L.tab_elems + W * F + i] = 0.f;
    }

    // ---------------------------------------------------------------- second forward pass
    // slack_i = K - D_i with K = T - Tot and D_i = max(D_{i-1}, cst_i - Pre_{i-1}), D_0 = 0
    // (a candidate with a bad level, K = NaN, gets its NaN row from the flush instead)
    const float Kc = tfin[cl] - pre;
    const float K = Kc == Kc ? Kc : 0.f;
    float D = 0.f, Pr = 0.f;
    win_load<ROWS16>(a, levels, g.tabt, 4, blocks, base, B, P, 0, s0);
    win_load<ROWS16>(a, levels, g.tabt, 4, blocks, base, B, P, nwin > 1 ? 1 : 0, s1);
    win_store<ROWS16>(a, lds, 0, tabt, 4, nullptr, addf, s0);
    lds_barrier();
    float *trow = tile + cl * (W + 1);
    auto scan_window = [&](int w, WinSet &ld, WinSet &cm) {
        const int buf = w & 1;
        win_load<ROWS16>(a, levels, g.tabt, 4, blocks, base, B, P, w + 2 < nwin ? w + 2 : nwin - 1, ld);
        const uint8_t *lrow = lvl0 + buf * L.lvl_buf + cl * L.lvl_pitch;
        const char *tb = reinterpret_cast<const char *>(tabt + buf * L.tab_elems);
        const ChainWinStep *rs = recs(buf);
        int k0, k1;
        win_range(a, lds, buf, ch, k0, k1);
        const int ng = (k1 - k0) >> 2;
        // group g of 4 steps, pipelined like the forward pass: its times are read while the
        // next group's level bytes and the records of the group after it are in flight
        auto stage = [&](WinGroup<FIXED> &A, WinGroup<FIXED> &Bn, WinGroup<FIXED> &C, int g) {
            float tt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                tt[i] = *reinterpret_cast<const float *>(tb + (((A.ct[i] >> 16) + A.lv[i]) << 2));
            Bn.levels(lrow);
            C.read(rs, k0 + 4 * (g + 2));
            win_issue_point();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                // (Pre summed as the forward pass sums it: table time, then fixed duration)
                D = fmaxf(D, A.cst[i] - Pr);
                Pr += tt[i];
                if (FIXED) Pr += A.dur[i];
                trow[A.ct[i] & 0xffffu] = K - D;
            }
        };
        WinGroup<FIXED> G0, G1, G2;
        G0.read(rs, k0);
        G1.read(rs, k0 + 4);
        G0.levels(lrow);
        for (int g = 0; g < ng; g += 3) {
            stage(G0, G1, G2, g);
            if (g + 1 >= ng) break;
            stage(G1, G2, G0, g + 1);
            if (g + 2 >= ng) break;
            stage(G2, G0, G1, g + 2);
        }
        if (w + 1 < nwin) win_store<ROWS16>(a, lds, buf ^ 1, tabt + (buf ^ 1) * L.tab_elems, 4, nullptr, addf, cm);
        lds_barrier();
        flush_tile(w);
        lds_barrier();
    };
    for (int w = 0; w < nwin; w += 2) {
        scan_window(w, s0, s1);
        if (w + 1 < nwin) scan_window(w + 1, s1, s0);
    }
}

// The two-pass chain scan (chains_windowed with slack) for the layouts where every window lies
// wholly inside the graph (P a multiple of W) and a thread holds at most four pieces of the slack
// tile: every window copy and every flush follows a per-thread plan fixed for the kernel, so the
// per-window work is the loads, the LDS stores, the flush stores and the barriers, with no bounds
// checks, category tests or zeroing.  The walk of each window is that of chains_windowed; a
// candidate with an invalid level gets its NaN row from the flush plan.
template <bool FIXED, int NT8>
__global__ void __launch_bounds__(kChainBlockThreads)
chains_scan_full(DevGraph g, DevChains c, WinArgs a, const uint4 *__restrict__ blocks,
                 const uint8_t *__restrict__ levels, int64_t B, float *__restrict__ To,
                 float *__restrict__ Eo, float *__restrict__ S) {
    extern __shared__ float4 smem[];
    char *lds = reinterpret_cast<char *>(smem);
    const int t = threadIdx.x, nt = blockDim.x;
    const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
    const int grp = wv / a.nc, ch = wv - grp * a.nc;
    const int lane = t & 63;
    const int cl = grp * 64 + lane;                               // candidate within the workgroup
    const int64_t base = static_cast<int64_t>(blockIdx.x) * a.NC;
    const int64_t gc = base + cl;
    const int W = a.W, F = a.F, nc = a.nc, nwin = c.nwin;
    const int32_t P = g.P;
    const WinLayout &L = a.L;
    const int64_t rows_left = B - base;
    uint8_t *lvl0 = reinterpret_cast<uint8_t *>(lds);             // [2][NC][W + 4] bytes
    uint32_t *bad = reinterpret_cast<uint32_t *>(lds + L.off_bad);
    float *tfin = reinterpret_cast<float *>(lds + L.off_tfin);
    float2 *tab2 = reinterpret_cast<float2 *>(lds + L.off_x);     // forward: [2][W + 1][F]
    float *tabt = reinterpret_cast<float *>(lds + L.off_x);       // second pass: [2][W + 1][F]
    float *tile = reinterpret_cast<float *>(lds + L.off_tile);    // second pass: [NC][W + 1]
    const uint32_t addf = (0x80u - static_cast<uint32_t>(F)) * 0x01010101u;
    // the bits of a byte that is >= F when F is a power of two
    const uint32_t hib = (F & (F - 1)) == 0 ? (0xffu & ~static_cast<uint32_t>(F - 1)) * 0x01010101u : 0u;
    auto recs = [&](int buf) {
        return reinterpret_cast<const ChainWinStep *>(lds + L.off_blk + buf * a.blk_bytes + 4 * a.hdr_words);
    };

    // ------------------------------------------------------------------ forward
    for (int i = t; i < a.NC; i += nt) {
        bad[i] = 0u;
        *reinterpret_cast<uint32_t *>(lvl0 + i * L.lvl_pitch + W) = 0u;
        *reinterpret_cast<uint32_t *>(lvl0 + L.lvl_buf + i * L.lvl_pitch + W) = 0u;
    }
    for (int i = t; i < F; i += nt) {
        tab2[W * F + i] = make_float2(0.f, 0.f);
        tab2[L.tab_elems + W * F + i] = make_float2(0.f, 0.f);
    }
    const uint32_t spare = L.total;                               // 1 KiB past the layout: spare slots
    WinPlan plan = win_plan<NT8>(a, 8, rows_left, P, spare);
    uint32_t badbits = 0u;
    const int64_t nrows = rows_left < a.NC ? rows_left : a.NC;
    WinBufs bf;
    bf.lvl = win_rsrc(levels + base * P, static_cast<uint32_t>(nrows * P));
    bf.tab = win_rsrc(g.tab, static_cast<uint32_t>(static_cast<int64_t>(P) * F * 8));
    bf.blk = win_rsrc(blocks, static_cast<uint32_t>(static_cast<int64_t>(nwin) * a.blk_bytes));
    bf.tab_win = W * F * 8;
    WinSet s0, s1;
    win_load_full<NT8>(a, plan, bf, 0, s0);
    win_load_full<NT8>(a, plan, bf, nwin > 1 ? 1 : 0, s1);
    lds_barrier();
    win_store_full<NT8>(plan, plan.dst0, lds, &badbits, addf, hib, s0);
    lds_barrier();
    float f = 0.f, pre = 0.f;
    double ed = 0.0;
    // window w from buffer buf = w & 1; `ld` takes window w + 2, `cm` holds window w + 1
    auto forward_window = [&](int w, int buf, WinSet &ld, WinSet &cm) {
        win_load_full<NT8>(a, plan, bf, w + 2 < nwin ? w + 2 : nwin - 1, ld);
        const uint8_t *lrow = lvl0 + buf * L.lvl_buf + cl * L.lvl_pitch;
        const char *tb = reinterpret_cast<const char *>(tab2 + buf * L.tab_elems);
        const ChainWinStep *rs = recs(buf);
        int k0, k1;
        win_range(a, lds, buf, ch, k0, k1);
        float eb = 0.f;
        const int ng = (k1 - k0) >> 2;
        auto stage = [&](WinGroup<FIXED> &A, WinGroup<FIXED> &Bn, WinGroup<FIXED> &C, int gi) {
            float2 te[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                te[i] = *reinterpret_cast<const float2 *>(tb + (((A.ct[i] >> 16) + A.lv[i]) << 3));
            Bn.levels(lrow);
            C.read(rs, k0 + 4 * (gi + 2));
            win_issue_point();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f = fmax_nonneg(f, A.cst[i]) + te[i].x;
                pre += te[i].x;
                if (FIXED) {
                    f += A.dur[i];
                    pre += A.dur[i];
                }
                eb += te[i].y;
            }
        };
        WinGroup<FIXED> G0, G1, G2;
        G0.read(rs, k0);
        G1.read(rs, k0 + 4);
        G0.levels(lrow);
        // fp32 energy blocks of at most 60 steps (15 groups, a whole number of rotations)
        for (int c0 = 0; c0 < ng; c0 += 15) {
            const int c1 = ng < c0 + 15 ? ng : c0 + 15;
            for (int gi = c0; gi < c1; gi += 3) {
                stage(G0, G1, G2, gi);
                if (gi + 1 >= c1) break;
                stage(G1, G2, G0, gi + 1);
                if (gi + 2 >= c1) break;
                stage(G2, G0, G1, gi + 2);
            }
            ed += static_cast<double>(eb);
            eb = 0.f;
        }
        // (after the last window: a copy of it into the idle buffer, which nothing reads)
        win_store_full<NT8>(plan, buf ? plan.dst0 : plan.dst1, lds, &badbits, addf, hib, cm);
        lds_barrier();
    };
    for (int w = 0; w < nwin; w += 2) {
        forward_window(w, 0, s0, s1);
        if (w + 1 < nwin) forward_window(w + 1, 1, s1, s0);
    }
    win_mark_bad(a, badbits, bad);
    // chains' makespans and energies -> the candidate's (chain order)
    double *esum = reinterpret_cast<double *>(lds + L.off_x);
    float *tsum = reinterpret_cast<float *>(lds + L.off_x + 8 * 64 * kWinMaxWaves);
    esum[wv * 64 + lane] = ed;
    tsum[wv * 64 + lane] = f;
    lds_barrier();
    if (ch == 0) {
        float T = c.t_const;
        double e = 0.0;
        for (int j = 0; j < nc; ++j) {
            T = fmaxf(T, tsum[(grp * nc + j) * 64 + lane]);
            e += esum[(grp * nc + j) * 64 + lane];
        }
        float E = static_cast<float>(e + static_cast<double>(g.static_power) * static_cast<double>(T));
        if (bad[cl]) {
            T = __builtin_nanf("");
            E = __builtin_nanf("");
        }
        tfin[cl] = T;
        if (gc < B) {
            To[gc] = T;
            Eo[gc] = E;
        }
    }
    lds_barrier();

    // ---------------------------------------------------------------- second forward pass
    // slack_i = K - D_i with K = T - Tot and D_i = max(D_{i-1}, cst_i - Pre_{i-1}) (see
    // chains_windowed); a candidate with an invalid level (K = NaN) gets NaN from the flush
    const FlushPlan fp = flush_plan(a, rows_left, P, tfin);
    const __amdgpu_buffer_rsrc_t srows = win_rsrc(S + base * P, static_cast<uint32_t>(nrows * P * 4));
    plan = win_plan<1>(a, 4, rows_left, P, spare);
    bf.tab = win_rsrc(g.tabt, static_cast<uint32_t>(static_cast<int64_t>(P) * F * 4));
    bf.tab_win = W * F * 4;
    for (int i = t; i < F; i += nt) {
        tabt[W * F + i] = 0.f;
        tabt[L.tab_elems + W * F + i] = 0.f;
    }
    const float Kc = tfin[cl] - pre;
    const float K = Kc == Kc ? Kc : 0.f;
    float D = 0.f, Pr = 0.f;
    win_load_full<1>(a, plan, bf, 0, s0);
    win_load_full<1>(a, plan, bf, nwin > 1 ? 1 : 0, s1);
    win_store_full<1>(plan, plan.dst0, lds, nullptr, addf, hib, s0);
    lds_barrier();
    float *trow = tile + cl * (W + 1);
    auto scan_window = [&](int w, int buf, WinSet &ld, WinSet &cm) {
        win_load_full<1>(a, plan, bf, w + 2 < nwin ? w + 2 : nwin - 1, ld);
        const uint8_t *lrow = lvl0 + buf * L.lvl_buf + cl * L.lvl_pitch;
        const char *tb = reinterpret_cast<const char *>(tabt + buf * L.tab_elems);
        const ChainWinStep *rs = recs(buf);
        int k0, k1;
        win_range(a, lds, buf, ch, k0, k1);
        const int ng = (k1 - k0) >> 2;
        auto stage = [&](WinGroup<FIXED> &A, WinGroup<FIXED> &Bn, WinGroup<FIXED> &C, int gi) {
            float tt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                tt[i] = *reinterpret_cast<const float *>(tb + (((A.ct[i] >> 16) + A.lv[i]) << 2));
            Bn.levels(lrow);
            C.read(rs, k0 + 4 * (gi + 2));
            win_issue_point();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                D = fmaxf(D, A.cst[i] - Pr);
                Pr += tt[i];
                if (FIXED) Pr += A.dur[i];
                trow[A.ct[i] & 0xffffu] = K - D;
            }
        };
        WinGroup<FIXED> G0, G1, G2;
        G0.read(rs, k0);
        G1.read(rs, k0 + 4);
        G0.levels(lrow);
        for (int gi = 0; gi < ng; gi += 3) {
            stage(G0, G1, G2, gi);
            if (gi + 1 >= ng) break;
            stage(G1, G2, G0, gi + 1);
            if (gi + 2 >= ng) break;
            stage(G2, G0, G1, gi + 2);
        }
        win_store_full<1>(plan, buf ? plan.dst0 : plan.dst1, lds, nullptr, addf, hib, cm);
        lds_barrier();
        flush_full(fp, srows, lds, w, a.wlog);
        lds_barrier();
    };
    for (int w = 0; w < nwin; w += 2) {
        scan_window(w, 0, s0, s1);
        if (w + 1 < nwin) scan_window(w + 1, 1, s1, s0);
    }
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

bool chain_window_fits(int32_t nc, int32_t F, int32_t W, int32_t blk_bytes, bool rows16, int32_t *groups) {
    if (nc < 1 || nc > kWinMaxWaves || F < 1 || F > 128 || W < 16 || W > 256 || blk_bytes % 16 != 0)
        return false;
    const int G = kWinMaxWaves / nc;
    const int NC = 64 * G, nthreads = 64 * G * nc;
    const WinLayout L = win_layout(W, NC, F, G * nc, blk_bytes);
    int sl, st8, st4, sb;
    if (L.total > kWinLds || !win_slots(W, NC, F, blk_bytes, nthreads, &sl, &st8, &st4, &sb)) return false;
    // rows that are not 16-byte aligned: one level piece per thread (its five dwords are held
    // from one window to the next)
    if (!rows16 && sl > 1) return false;
    *groups = G;
    return true;
}

bool chains_scan_ok(const DevChains &c, const uint8_t *levels, const float *slack) {
    return slack && chains_windowed_ok(c, levels, slack);
}

bool chains_scan_full_ok(const DevChains &c, const uint8_t *levels, const float *slack) {
    return c.full && chains_scan_ok(c, levels, slack);
}

bool chains_windowed_ok(const DevChains &c, const uint8_t *levels, const float *slack) {
    return c.win > 0 && reinterpret_cast<uintptr_t>(levels) % 16 == 0 &&
           reinterpret_cast<uintptr_t>(slack) % 16 == 0;
}

namespace {
int64_t win_grid(const DevChains &c, int64_t B) {
    const int64_t NC = 64 * static_cast<int64_t>(c.groups);
    return (B + NC - 1) / NC;
}
}  // namespace

size_t chains_scratch_bytes(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                            const float *slack_ptr) {
    const bool slack = slack_ptr != nullptr;
    // windowed layout: the makespan and energy when the caller does not take them
    if (chains_windowed_ok(c, levels, slack_ptr)) return 2 * round256(static_cast<size_t>(B) * sizeof(float));
    const size_t lanes = static_cast<size_t>(chain_grid(c, B)) * kChainBlockThreads;
    const size_t ck = slack ? round256(static_cast<size_t>(c.len / K) * lanes * sizeof(float)) : 0;
    const size_t tmp = slack && staged_ok(g, c) && g.P % 4 == 0
                           ? round256(static_cast<size_t>(B) * (static_cast<size_t>(c.len) << c.lane_log) * sizeof(float))
                           : 0;
    return ck + tmp + 2 * round256(static_cast<size_t>(B) * sizeof(float));
}

namespace {
template <bool SLACK, bool FIXED, bool ROWS16>
hipError_t launch_windowed_kernel(dim3 gd, dim3 bd, size_t lds, hipStream_t s, const DevGraph &g,
                                  const DevChains &c, const WinArgs &a, const uint8_t *levels, int64_t B,
                                  float *T, float *E, float *S) {
    // the dynamic LDS limit is raised once per device (the caller made the graph's device current)
    static std::atomic<uint64_t> done{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev < 64 ? uint64_t{1} << dev : 0;
    if (!bit || !(done.load(std::memory_order_acquire) & bit)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&chains_windowed<SLACK, FIXED, ROWS16>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kWinLds));
        if (e != hipSuccess) return e;
        done.fetch_or(bit, std::memory_order_acq_rel);
    }
    hipLaunchKernelGGL((chains_windowed<SLACK, FIXED, ROWS16>), gd, bd, lds, s, g, c, a, c.blocks, levels, B, T,
                       E, S);
    return hipGetLastError();
}

template <bool FIXED, int NT8>
hipError_t launch_scan_full_kernel(dim3 gd, dim3 bd, size_t lds, hipStream_t s, const DevGraph &g,
                                   const DevChains &c, const WinArgs &a, const uint8_t *levels, int64_t B,
                                   float *T, float *E, float *S) {
    static std::atomic<uint64_t> done{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev < 64 ? uint64_t{1} << dev : 0;
    if (!bit || !(done.load(std::memory_order_acquire) & bit)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void *>(&chains_scan_full<FIXED, NT8>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kWinLds + kWinSpare));
        if (e != hipSuccess) return e;
        done.fetch_or(bit, std::memory_order_acq_rel);
    }
    hipLaunchKernelGGL((chains_scan_full<FIXED, NT8>), gd, bd, lds + kWinSpare, s, g, c, a, c.blocks, levels, B, T,
                       E, S);
    return hipGetLastError();
}

hipError_t launch_windowed(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                           float *T, float *E, float *slack, const SelTargets &tg, void *scratch,
                           hipStream_t s) {
    WinArgs a;
    a.W = c.win;
    a.wlog = 0;
    while ((1 << a.wlog) < a.W) ++a.wlog;
    a.nc = c.nc;
    a.NC = 64 * c.groups;
    a.F = g.F;
    a.blk_bytes = c.blk_bytes;
    a.hdr_words = c.hdr_words;
    win_slots(a.W, a.NC, a.F, a.blk_bytes, 64 * c.groups * c.nc, &a.slots_lvl, &a.slots_tab8, &a.slots_tab4,
              &a.slots_blk);
    a.L = win_layout(a.W, a.NC, a.F, c.groups * c.nc, c.blk_bytes);
    const int64_t grid = win_grid(c, B);
    char *p = static_cast<char *>(scratch);
    const size_t vec = round256(static_cast<size_t>(B) * sizeof(float));
    float *Ts = T ? T : reinterpret_cast<float *>(p);
    float *Es = E ? E : reinterpret_cast<float *>(p + vec);
    const dim3 gd(static_cast<unsigned>(grid)), bd(static_cast<unsigned>(64 * c.groups * c.nc));
    const size_t lds = a.L.total;
    hipError_t e;
#define EMO_WIN_ARGS gd, bd, lds, s, g, c, a, levels, B, Ts, Es, slack
    if (slack && c.full) {
        // one or two 16-byte forward table pieces per thread (c.full guarantees the rest of the
        // slot layout: one level piece, one block piece, one second-pass table piece)
        const bool two = a.slots_tab8 == 2;
        e = c.fixed ? (two ? launch_scan_full_kernel<true, 2>(gd, bd, lds, s, g, c, a, levels, B, Ts, Es, slack)
                           : launch_scan_full_kernel<true, 1>(gd, bd, lds, s, g, c, a, levels, B, Ts, Es, slack))
                    : (two ? launch_scan_full_kernel<false, 2>(gd, bd, lds, s, g, c, a, levels, B, Ts, Es, slack)
                           : launch_scan_full_kernel<false, 1>(gd, bd, lds, s, g, c, a, levels, B, Ts, Es, slack));
    } else if (g.P % 16 == 0) {
        e = slack ? (c.fixed ? launch_windowed_kernel<true, true, true>(EMO_WIN_ARGS)
                             : launch_windowed_kernel<true, false, true>(EMO_WIN_ARGS))
                  : (c.fixed ? launch_windowed_kernel<false, true, true>(EMO_WIN_ARGS)
                             : launch_windowed_kernel<false, false, true>(EMO_WIN_ARGS));
    } else {
        e = slack ? (c.fixed ? launch_windowed_kernel<true, true, false>(EMO_WIN_ARGS)
                             : launch_windowed_kernel<true, false, false>(EMO_WIN_ARGS))
                  : (c.fixed ? launch_windowed_kernel<false, true, false>(EMO_WIN_ARGS)
                             : launch_windowed_kernel<false, false, false>(EMO_WIN_ARGS));
    }
#undef EMO_WIN_ARGS
    if (e == hipSuccess && tg.n) e = launch_select_results(Ts, Es, B, tg, s);
    return e;
}
}  // namespace

hipError_t launch_chains(const DevGraph &g, const DevChains &c, const uint8_t *levels, int64_t B,
                         float *T, float *E, float *slack, const SelTargets &tg, void *scratch,
                         hipStream_t s) {
    if (chains_windowed_ok(c, levels, slack)) return launch_windowed(g, c, levels, B, T, E, slack, tg, scratch, s);
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
    if (e == hipSuccess && tg.n) e = launch_select_results(Ts, Es, B, tg, s);
    return e;
}

}  // namespace emo
