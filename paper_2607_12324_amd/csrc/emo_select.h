// Device-side selection (Eq. 4): feasibility mask and least-energy feasible candidate.
//
// Shared by the precompiled kernels and by the graph-specialised kernels compiled at run time
// (its text is embedded into the library and prepended to the generated source), so it
// includes no headers and uses only HIP built-ins.
//
// The caller's result record (24 bytes, see emo_selection) is the accumulator while a
// selection runs:
//   bytes 0..7   u64 key = (fp32 bits of E) << 32 | candidate; energies are >= 0, so the bit
//                pattern orders like the value and equal energies order by index
//   bytes 8..11  u32 number of blocks done; the last block to finish writes the final record
//   bytes 16..23 u64 number of feasible candidates
#pragma once

#ifndef EMO_BLOCK
#define EMO_BLOCK 256
#endif
#define EMO_WAVE 64
#define EMO_WAVES_PER_BLOCK (EMO_BLOCK / EMO_WAVE)

struct EmoAcc {
    unsigned long long key;
    unsigned int done;
    unsigned int pad;
    unsigned long long count;
};

struct EmoSel {
    long long index;
    float energy;
    float makespan;
    long long num_feasible;
};

__device__ __forceinline__ unsigned long long emo_wave_min_u64(unsigned long long v) {
    for (int off = EMO_WAVE / 2; off > 0; off >>= 1) {
        unsigned long long o = __shfl_xor(v, off, EMO_WAVE);
        v = o < v ? o : v;
    }
    return v;
}

// Reduces feasibility, count and key over the block and the grid.  Returns true in every
// thread of the last block to finish, with *key_out / *count_out holding the grid results.
// Must be called by every thread of the block.
__device__ bool emo_select_reduce(bool active, float T, float E, long long c, long long B,
                                  float target, unsigned int *mask, void *res,
                                  unsigned long long *key_out, unsigned long long *count_out) {
    __shared__ unsigned long long s_key[EMO_WAVES_PER_BLOCK];
    __shared__ unsigned int s_cnt[EMO_WAVES_PER_BLOCK];
    __shared__ unsigned long long s_res[2];
    __shared__ int s_last;
    const bool feas = active && (T <= target);   // false for NaN
    const unsigned long long bal = __ballot(feas);
    const int lane = threadIdx.x % EMO_WAVE;
    const int wave = threadIdx.x / EMO_WAVE;
    const long long wbase = (long long)blockIdx.x * EMO_BLOCK + wave * EMO_WAVE;
    if (mask && lane == 0 && wbase < B) {
        const long long nwords = (B + 31) / 32;
        const long long w = wbase / 32;
        mask[w] = (unsigned int)bal;
        if (w + 1 < nwords) mask[w + 1] = (unsigned int)(bal >> 32);
    }
    unsigned long long key = feas ? (((unsigned long long)__float_as_uint(E)) << 32) |
                                        (unsigned long long)(unsigned int)c
                                  : ~0ull;
    key = emo_wave_min_u64(key);
    if (lane == 0) {
        s_key[wave] = key;
        s_cnt[wave] = (unsigned int)__popcll(bal);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long bk = s_key[0];
        unsigned long long bc = s_cnt[0];
        for (int w = 1; w < EMO_WAVES_PER_BLOCK; ++w) {
            bk = s_key[w] < bk ? s_key[w] : bk;
            bc += s_cnt[w];
        }
        EmoAcc *a = (EmoAcc *)res;
        if (bk != ~0ull) atomicMin(&a->key, bk);
        if (bc) atomicAdd(&a->count, bc);
        __threadfence();
        const unsigned int ticket = atomicAdd(&a->done, 1u);
        s_last = ticket == gridDim.x - 1;
        if (s_last) {
            __threadfence();
            s_res[0] = atomicAdd(&a->key, 0ull);
            s_res[1] = atomicAdd(&a->count, 0ull);
        }
    }
    __syncthreads();
    *key_out = s_res[0];
    *count_out = s_res[1];
    return s_last != 0;
}

// Winner index from a grid key (0 when nothing is feasible, so that it can be re-evaluated
// safely).
__device__ __forceinline__ long long emo_key_index(unsigned long long key) {
    return key == ~0ull ? 0 : (long long)(key & 0xffffffffull);
}

__device__ __forceinline__ void emo_write_selection(void *res, unsigned long long key,
                                                    unsigned long long count, float T_winner) {
    EmoSel *r = (EmoSel *)res;
    if (key == ~0ull) {
        r->index = -1;
        r->energy = __builtin_nanf("");
        r->makespan = __builtin_nanf("");
    } else {
        r->index = (long long)(key & 0xffffffffull);
        r->energy = __uint_as_float((unsigned int)(key >> 32));
        r->makespan = T_winner;
    }
    r->num_feasible = (long long)count;
}
