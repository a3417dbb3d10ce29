// Device kernels of the policy search (Alg. 2, Sec. IV-F) with one frequency interval per pack.
//
// A stage of the dynamic program sets the level of one pack p in every stored policy: the
// stored states (one per makespan bucket) are S x F candidate rows (each stored policy with
// every level f at p), the candidates are evaluated by the batch evaluator (Alg. 1), each
// bucket keeps the candidate with the least key (fp32 energy bits << 32 | candidate index): the least energy,
// and among equal energies the first candidate in the order (state, level), as a sequential
// "replace when strictly lower" walk over the states in bucket order would keep; the winners are
// then written out directly as the next stage's candidate rows.
#include <hip/hip_runtime.h>

#include <algorithm>

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

// dp[0] = {P_0}: row0 (P_0, evaluated: T[0], E[0]) is the only stored policy.  Without packs it
// is the final state (state, key, Tst); otherwise it is expanded into the F candidate rows of
// the first stage (level f at pack p), its key marks it stored, and the first stage's output
// keys are cleared.  (dp[0] keeps P_0 whatever its makespan: the initialisation of Alg. 2 does
// not test the constraint.)
__global__ void dp_seed(const uint8_t *__restrict__ row0, int32_t P, int32_t F, int32_t p,
                        const float *__restrict__ T, const float *__restrict__ E,
                        uint8_t *__restrict__ rows, uint8_t *__restrict__ state,
                        unsigned long long *__restrict__ key, float *__restrict__ Tst,
                        unsigned long long *__restrict__ out_keys, int64_t NB) {
    const int64_t n = p >= 0 ? static_cast<int64_t>(F) * P : 0;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int32_t f = static_cast<int32_t>(i / P), col = static_cast<int32_t>(i - static_cast<int64_t>(f) * P);
        rows[i] = col == p ? static_cast<uint8_t>(f) : row0[col];
    }
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < P;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        state[i] = row0[i];
    for (int64_t b = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; b < NB;
         b += static_cast<int64_t>(gridDim.x) * blockDim.x)
        out_keys[b] = kEmptyKey;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        key[0] = static_cast<unsigned long long>(__float_as_uint(E[0])) << 32;
        Tst[0] = T[0];
    }
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

// After the bucket step of a stage: the winning candidate of each bucket b becomes stored
// policy b.  With a next pack p_next >= 0 it is expanded at once into that stage's candidate
// rows next_rows[b * F + f] (level f at p_next); after the last stage it is copied to state[b]
// with its makespan Tst[b].  Also clears done_keys (the keys of this stage's source states, no
// longer read), which the next stage's bucket step fills.
// Grid: x covers a row in pieces (16 bytes when P is a multiple of 16, else single bytes), y the
// output rows (next_rows or state); row y of the expansion is bucket y / F at level y % F.
__global__ void dp_advance(const uint8_t *__restrict__ rows, const float *__restrict__ T,
                           const unsigned long long *__restrict__ keys, int64_t NB, int32_t P,
                           int32_t F, int32_t p_next, uint8_t *__restrict__ next_rows,
                           uint8_t *__restrict__ state, float *__restrict__ Tst,
                           unsigned long long *__restrict__ done_keys) {
    const int64_t nrows = p_next >= 0 ? NB * F : NB;
    const bool vec = P % 16 == 0;
    const int32_t npiece = vec ? P / 16 : P;
    const int32_t x = static_cast<int32_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x < npiece) {
        for (int64_t y = blockIdx.y; y < nrows; y += gridDim.y) {
            const int64_t b = p_next >= 0 ? y / F : y;
            const unsigned long long k = keys[b];
            if (k == kEmptyKey) continue;
            const int64_t c = static_cast<int64_t>(k & 0xffffffffull);
            const uint8_t f = static_cast<uint8_t>(y - b * F);
            uint8_t *dst = (p_next >= 0 ? next_rows : state) + y * P;
            const uint8_t *src = rows + c * P;
            if (vec) {
                uint4 v = reinterpret_cast<const uint4 *>(src)[x];
                const int32_t o = p_next - 16 * x;   // the pack's byte within this piece, if any
                if (p_next >= 0 && o >= 0 && o < 16) {
                    uint32_t *w = o < 4 ? &v.x : (o < 8 ? &v.y : (o < 12 ? &v.z : &v.w));
                    const int sh = 8 * (o & 3);
                    *w = (*w & ~(0xffu << sh)) | (static_cast<uint32_t>(f) << sh);
                }
                reinterpret_cast<uint4 *>(dst)[x] = v;
            } else {
                dst[x] = x == p_next ? f : src[x];
            }
        }
    }
    if (blockIdx.x == 0 && blockIdx.y == 0)
        for (int64_t b = threadIdx.x; b < NB; b += blockDim.x) {
            const unsigned long long k = keys[b];
            if (k != kEmptyKey) Tst[b] = T[k & 0xffffffffull];
            done_keys[b] = kEmptyKey;
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

hipError_t dp_launch_seed(const uint8_t *row0, int32_t P, int32_t F, int32_t p, const float *T,
                          const float *E, uint8_t *rows, uint8_t *state, unsigned long long *key,
                          float *Tst, unsigned long long *out_keys, int64_t NB, hipStream_t s) {
    const int64_t n = std::max<int64_t>(std::max<int64_t>(static_cast<int64_t>(F) * P, NB), 1);
    dp_seed<<<blocks_for(n), kThreads, 0, s>>>(row0, P, F, p, T, E, rows, state, key, Tst, out_keys, NB);
    return hipGetLastError();
}

hipError_t dp_launch_bucket(const float *T, const float *E, const unsigned long long *src_keys,
                            int64_t B, int32_t F, float tmax, double q, int64_t bmin, int64_t NB,
                            unsigned long long *keys, hipStream_t s) {
    dp_bucket<<<blocks_for(B), kThreads, 0, s>>>(T, E, src_keys, B, F, tmax, q, bmin, NB, keys);
    return hipGetLastError();
}

hipError_t dp_launch_advance(const uint8_t *rows, const float *T, const unsigned long long *keys,
                             int64_t NB, int32_t P, int32_t F, int32_t p_next, uint8_t *next_rows,
                             uint8_t *state, float *Tst, unsigned long long *done_keys, hipStream_t s) {
    const int64_t nrows = p_next >= 0 ? NB * F : NB;
    const int64_t npiece = P % 16 == 0 ? P / 16 : P;
    const dim3 grid(static_cast<unsigned>(std::max<int64_t>((npiece + kThreads - 1) / kThreads, 1)),
                    static_cast<unsigned>(std::min<int64_t>(std::max<int64_t>(nrows, 1), 65535)));
    dp_advance<<<grid, kThreads, 0, s>>>(rows, T, keys, NB, P, F, p_next, next_rows, state, Tst, done_keys);
    return hipGetLastError();
}

hipError_t dp_launch_final(const uint8_t *states, const unsigned long long *keys, const float *Tst,
                           int64_t S, int32_t P, float tmax, double q, uint8_t *best,
                           emo_selection *res, hipStream_t s) {
    dp_final<<<1, kThreads, 0, s>>>(states, keys, Tst, S, P, tmax, q, best, res);
    return hipGetLastError();
}

}  // namespace emo
