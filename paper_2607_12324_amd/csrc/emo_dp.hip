// Device kernels of the policy search (Alg. 2, Sec. IV-F) with one frequency interval per pack.
//
// A stage of the dynamic program sets the level of one pack p in every stored policy: the
// stored states (one per makespan bucket, a level row each) are expanded into S x F candidate
// rows, the candidates are evaluated by the batch evaluator (Alg. 1), and each bucket keeps the
// candidate with the least key (fp32 energy bits << 32 | candidate index): the least energy,
// and among equal energies the first candidate in the order (state, level), as a sequential
// "replace when strictly lower" walk over the states in bucket order would keep.
#include <hip/hip_runtime.h>

#include "emo_internal.h"

namespace emo {
namespace {

constexpr unsigned long long kEmptyKey = ~0ull;
constexpr int kThreads = 256;

unsigned blocks_for(int64_t n) {
    const int64_t b = (n + kThreads - 1) / kThreads;
    return static_cast<unsigned>(b < 1 ? 1 : (b > 65536 ? 65536 : b));
}

// The policy P_0 (level F-1 everywhere) as candidate row 0.
__global__ void dp_default_row(uint8_t *__restrict__ row, int32_t P, uint8_t top) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < P; i += gridDim.x * blockDim.x) row[i] = top;
}

// dp[0] = {P_0}: one state holding row 0 with P_0's makespan and energy (kept whatever the
// makespan: the initialisation of Alg. 2 does not test the constraint).
__global__ void dp_init_state(const uint8_t *__restrict__ row, int32_t P, const float *__restrict__ T,
                              const float *__restrict__ E, uint8_t *__restrict__ state,
                              unsigned long long *__restrict__ key, float *__restrict__ Tst) {
    for (int32_t i = threadIdx.x; i < P; i += blockDim.x) state[i] = row[i];
    if (threadIdx.x == 0) {
        key[0] = (static_cast<unsigned long long>(__float_as_uint(E[0])) << 32);
        Tst[0] = T[0];
    }
}

// rows[s * F + f] = state s with level f at pack p.  States that hold no policy are expanded
// as well (their rows are evaluated and then ignored), so the grid does not depend on them.
__global__ void dp_expand(const uint8_t *__restrict__ states, int64_t S, int32_t P, int32_t F,
                          int32_t p, uint8_t *__restrict__ rows) {
    const int64_t n = S * F * P;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = i / P;
        const int32_t col = static_cast<int32_t>(i - r * P);
        const int64_t s = r / F;
        rows[i] = col == p ? static_cast<uint8_t>(r - s * F) : states[s * P + col];
    }
}

__global__ void dp_clear_keys(unsigned long long *__restrict__ keys, int64_t n) {
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        keys[i] = kEmptyKey;
}

// Candidate c (from state c / F) with makespan T[c] <= tmax proposes itself for bucket
// floor(T / q) - bmin (in double precision); the least key of a bucket wins.
__global__ void dp_bucket(const float *__restrict__ T, const float *__restrict__ E,
                          const unsigned long long *__restrict__ src_keys, int64_t B, int32_t F,
                          float tmax, double q, int64_t bmin, int64_t NB,
                          unsigned long long *__restrict__ keys) {
    for (int64_t c = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; c < B;
         c += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (src_keys[c / F] == kEmptyKey) continue;
        const float t = T[c];
        if (!(t <= tmax)) continue;   // also drops NaN
        const int64_t b = static_cast<int64_t>(floor(static_cast<double>(t) / q)) - bmin;
        if (b < 0 || b >= NB) continue;
        const unsigned long long k =
            (static_cast<unsigned long long>(__float_as_uint(E[c])) << 32) | static_cast<unsigned long long>(c);
        atomicMin(&keys[b], k);
    }
}

// dst[b] = the winning candidate row of bucket b, Tst[b] its makespan.
__global__ void dp_gather(const uint8_t *__restrict__ rows, const float *__restrict__ T,
                          const unsigned long long *__restrict__ keys, int64_t NB, int32_t P,
                          uint8_t *__restrict__ dst, float *__restrict__ Tst) {
    const int64_t n = NB * P;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t b = i / P;
        const unsigned long long k = keys[b];
        if (k == kEmptyKey) continue;
        dst[i] = rows[static_cast<int64_t>(k & 0xffffffffull) * P + (i - b * P)];
    }
    for (int64_t b = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; b < NB;
         b += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const unsigned long long k = keys[b];
        if (k != kEmptyKey) Tst[b] = T[k & 0xffffffffull];
    }
}

// The least (energy, bucket) over the stored states whose makespan meets tmax: its level row
// to best, and {floor(makespan / q) or -1, energy, makespan, number of such states} to res.
// One workgroup.
__global__ void __launch_bounds__(kThreads)
dp_final(const uint8_t *__restrict__ states, const unsigned long long *__restrict__ keys,
         const float *__restrict__ Tst, int64_t S, int32_t P, float tmax, double q,
         uint8_t *__restrict__ best, emo_selection *__restrict__ res) {
    __shared__ unsigned long long s_key[kThreads];
    __shared__ long long s_cnt[kThreads];
    unsigned long long mine = kEmptyKey;
    long long cnt = 0;
    for (int64_t b = threadIdx.x; b < S; b += kThreads) {
        const unsigned long long k = keys[b];
        if (k == kEmptyKey || !(Tst[b] <= tmax)) continue;
        ++cnt;
        const unsigned long long kb = (k & 0xffffffff00000000ull) | static_cast<unsigned long long>(b);
        mine = kb < mine ? kb : mine;
    }
    s_key[threadIdx.x] = mine;
    s_cnt[threadIdx.x] = cnt;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) {
            const unsigned long long o = s_key[threadIdx.x + w];
            if (o < s_key[threadIdx.x]) s_key[threadIdx.x] = o;
            s_cnt[threadIdx.x] += s_cnt[threadIdx.x + w];
        }
        __syncthreads();
    }
    const unsigned long long kbest = s_key[0];
    if (kbest != kEmptyKey) {
        const int64_t b = static_cast<int64_t>(kbest & 0xffffffffull);
        for (int32_t i = threadIdx.x; i < P; i += kThreads) best[i] = states[b * P + i];
    }
    if (threadIdx.x == 0) {
        if (kbest == kEmptyKey) {
            res->index = -1;
            res->energy = __builtin_nanf("");
            res->makespan = __builtin_nanf("");
        } else {
            const int64_t b = static_cast<int64_t>(kbest & 0xffffffffull);
            res->index = static_cast<int64_t>(floor(static_cast<double>(Tst[b]) / q));
            res->energy = __uint_as_float(static_cast<unsigned int>(kbest >> 32));
            res->makespan = Tst[b];
        }
        res->num_feasible = s_cnt[0];
    }
}

}  // namespace

hipError_t dp_launch_default_row(uint8_t *row, int32_t P, int32_t F, hipStream_t s) {
    if (P == 0) return hipSuccess;
    dp_default_row<<<blocks_for(P), kThreads, 0, s>>>(row, P, static_cast<uint8_t>(F - 1));
    return hipGetLastError();
}

hipError_t dp_launch_init_state(const uint8_t *row, int32_t P, const float *T, const float *E,
                                uint8_t *state, unsigned long long *key, float *Tst, hipStream_t s) {
    dp_init_state<<<1, kThreads, 0, s>>>(row, P, T, E, state, key, Tst);
    return hipGetLastError();
}

hipError_t dp_launch_expand(const uint8_t *states, int64_t S, int32_t P, int32_t F, int32_t p,
                            uint8_t *rows, hipStream_t s) {
    dp_expand<<<blocks_for(S * F * P), kThreads, 0, s>>>(states, S, P, F, p, rows);
    return hipGetLastError();
}

hipError_t dp_launch_select(const float *T, const float *E, const unsigned long long *src_keys,
                            int64_t B, int32_t F, float tmax, double q, int64_t bmin, int64_t NB,
                            unsigned long long *keys, hipStream_t s) {
    dp_clear_keys<<<blocks_for(NB), kThreads, 0, s>>>(keys, NB);
    dp_bucket<<<blocks_for(B), kThreads, 0, s>>>(T, E, src_keys, B, F, tmax, q, bmin, NB, keys);
    return hipGetLastError();
}

hipError_t dp_launch_gather(const uint8_t *rows, const float *T, const unsigned long long *keys,
                            int64_t NB, int32_t P, uint8_t *dst, float *Tst, hipStream_t s) {
    dp_gather<<<blocks_for(NB * (P > 0 ? P : 1)), kThreads, 0, s>>>(rows, T, keys, NB, P, dst, Tst);
    return hipGetLastError();
}

hipError_t dp_launch_final(const uint8_t *states, const unsigned long long *keys, const float *Tst,
                           int64_t S, int32_t P, float tmax, double q, uint8_t *best,
                           emo_selection *res, hipStream_t s) {
    dp_final<<<1, kThreads, 0, s>>>(states, keys, Tst, S, P, tmax, q, best, res);
    return hipGetLastError();
}

}  // namespace emo
