// Device-side selection (Eq. 4): feasibility mask and least-energy feasible candidate.
//
// Shared by the precompiled kernels and by the graph-specialised kernels compiled at run time
// (its text is embedded into the library and prepended to the generated source), so it
// includes no headers and uses only HIP built-ins.
//
// Two stages, with no atomics (thousands of blocks updating one address would serialise):
//   1. for every group of EMO_BLOCK consecutive candidates, the workgroup that evaluates it
//      writes the mask bits of its candidates and one partial record: its least key, its number
//      of feasible candidates and the makespan of the candidate holding that key;
//   2. one workgroup reduces the partial records and writes the emo_selection record (a kernel
//      of the precompiled library, launched after the evaluating kernel).
// The key of a feasible candidate c is (fp32 bits of its energy) << 32 | c.  Energies are
// >= 0, so the bit pattern orders like the value and equal energies order by index; an
// infeasible candidate has the key ~0.
#pragma once

#ifndef EMO_BLOCK
#define EMO_BLOCK 256
#endif
#define EMO_WAVE 64
#define EMO_WAVES_PER_BLOCK (EMO_BLOCK / EMO_WAVE)

struct EmoPartial {
    unsigned long long key;
    unsigned int count;
    float makespan;
};

struct EmoSel {
    long long index;
    float energy;
    float makespan;
    long long num_feasible;
};

// Mask words and partial records are stored through global (address space 1) pointers: a
// pointer taken from the targets' argument array with a run-time index is otherwise generic,
// and its flat stores would also count against the LDS wait counter.
#define EMO_SEL_GLOBAL(T, p) ((__attribute__((address_space(1))) T *)(p))
typedef unsigned int emo_sel_u4 __attribute__((ext_vector_type(4)));

// Least key over the wave, carrying the makespan of its candidate.
__device__ __forceinline__ void emo_wave_min_key(unsigned long long *key, float *T) {
    for (int off = EMO_WAVE / 2; off > 0; off >>= 1) {
        const unsigned long long ok = __shfl_xor(*key, off, EMO_WAVE);
        const float oT = __shfl_xor(*T, off, EMO_WAVE);
        if (ok < *key) {
            *key = ok;
            *T = oT;
        }
    }
}

// Stage 1 for the workgroup's current group of EMO_BLOCK consecutive candidates (group index
// `group`, candidates group * EMO_BLOCK + threadIdx.x).  Must be called by every thread of the
// workgroup.  `part` (one record per group) and `mask` may be NULL.
__device__ void emo_select_block(long long group, bool active, float T, float E, long long c,
                                 long long B, float target, unsigned int *mask, EmoPartial *part) {
    __shared__ unsigned long long s_key[EMO_WAVES_PER_BLOCK];
    __shared__ float s_T[EMO_WAVES_PER_BLOCK];
    __shared__ unsigned int s_cnt[EMO_WAVES_PER_BLOCK];
    const bool feas = active && (T <= target);   // false for NaN
    const unsigned long long bal = __ballot(feas);
    const int lane = threadIdx.x % EMO_WAVE;
    const int wave = threadIdx.x / EMO_WAVE;
    const long long wbase = group * EMO_BLOCK + wave * EMO_WAVE;
    if (mask && lane == 0 && wbase < B) {
        const long long nwords = (B + 31) / 32;
        const long long w = wbase / 32;
        EMO_SEL_GLOBAL(unsigned int, mask)[w] = (unsigned int)bal;
        if (w + 1 < nwords) EMO_SEL_GLOBAL(unsigned int, mask)[w + 1] = (unsigned int)(bal >> 32);
    }
    if (!part) return;
    unsigned long long key = feas ? (((unsigned long long)__float_as_uint(E)) << 32) |
                                        (unsigned long long)(unsigned int)c
                                  : ~0ull;
    float kT = T;
    emo_wave_min_key(&key, &kT);
    if (lane == 0) {
        s_key[wave] = key;
        s_T[wave] = kT;
        s_cnt[wave] = (unsigned int)__popcll(bal);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        EmoPartial p;
        p.key = s_key[0];
        p.makespan = s_T[0];
        p.count = s_cnt[0];
        for (int w = 1; w < EMO_WAVES_PER_BLOCK; ++w) {
            if (s_key[w] < p.key) {
                p.key = s_key[w];
                p.makespan = s_T[w];
            }
            p.count += s_cnt[w];
        }
        // one 16-byte store in the record's layout: key (low word first), count, makespan
        const emo_sel_u4 v = {(unsigned int)p.key, (unsigned int)(p.key >> 32), p.count,
                              __float_as_uint(p.makespan)};
        *EMO_SEL_GLOBAL(emo_sel_u4, part + group) = v;
    }
}

// The latency targets of one evaluation (Eq. 4 at each of them): the feasibility mask of target
// k goes to mask[k] (when not NULL) and its per-group partial records to part + k * nparts (all
// targets, when part is not NULL).  n = 0: no mask and no selection.
#define EMO_MAX_TARGETS 8
struct EmoTargets {
    int n;
    int pad;
    long long nparts;
    EmoPartial *part;
    float t[EMO_MAX_TARGETS];
    unsigned int *mask[EMO_MAX_TARGETS];
};

// Stage 1 for every target of `tg` (see emo_select_block; called by every thread of the
// workgroup, the targets one after another).
__device__ void emo_select_all(long long group, bool active, float T, float E, long long c,
                               long long B, const EmoTargets &tg) {
    for (int k = 0; k < tg.n; ++k) {
        // the previous target's records in LDS have been read before they are overwritten
        if (k > 0 && tg.part) __syncthreads();
        emo_select_block(group, active, T, E, c, B, tg.t[k], tg.mask[k],
                         tg.part ? tg.part + k * tg.nparts : (EmoPartial *)0);
    }
    // thread 0 has read the last target's per-wave values before any wave of this workgroup
    // goes on (a workgroup that walks several groups writes them again for the next group)
    if (tg.part) __syncthreads();
}

