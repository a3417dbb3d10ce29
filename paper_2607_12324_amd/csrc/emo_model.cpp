// Microbenchmark pack model (Sec. IV-E, Eq. 6-7), a host-only load-time pass: non-negative
// least squares of each pack's metric vector against the suite's metric matrix, then the
// pack's latency/energy tables as the weighted sums of the suite's.
//
// The NNLS solver is the active-set method of Lawson and Hanson (Solving Least Squares
// Problems, 1974, ch. 23): add the free weight of largest positive gradient to the passive set,
// solve least squares on the passive columns, and step back to the boundary while a passive
// weight would turn non-positive.  Here each passive-set subproblem is solved by Householder QR of the passive
// columns of B (Lawson and Hanson's own form), which keeps the conditioning of B rather than
// of B^T B: suites with fewer metrics than benchmarks are rank-deficient.  All arithmetic is
// double; packs are independent and split over host threads.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <atomic>
#include <thread>
#include <vector>

#include "emo.h"
#include "emo_internal.h"

namespace {

constexpr int kMaxBench = 64;

emo_status fail(emo_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    return emo::report(s, buf);
}

constexpr int kMaxMetrics = 256;

// Least squares on the passive columns S (k of them): z = argmin ||B[:, S] z - b|| by
// Householder QR of the n x k column block.  Returns false when a column is numerically
// dependent on the ones before it (|R_jj| <= 1e-10 of the column's norm).
bool solve_passive(const double *B, int n, int m, const double *b, const int *S, int k, double *z) {
    static thread_local std::vector<double> A, r;
    A.resize(size_t(n) * k);
    r.assign(b, b + n);
    double norm0[kMaxBench];
    for (int j = 0; j < k; ++j) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) {
            A[size_t(i) * k + j] = B[size_t(i) * m + S[j]];
            s += A[size_t(i) * k + j] * A[size_t(i) * k + j];
        }
        norm0[j] = std::sqrt(s);
    }
    if (k > n) return false;
    double diag[kMaxBench];
    for (int j = 0; j < k; ++j) {
        double s = 0.0;
        for (int i = j; i < n; ++i) s += A[size_t(i) * k + j] * A[size_t(i) * k + j];
        const double nrm = std::sqrt(s);
        if (!(nrm > 1e-10 * norm0[j])) return false;
        const double alpha = A[size_t(j) * k + j] > 0.0 ? -nrm : nrm;
        // reflector v = a_j - alpha e_j, stored in place; H = I - 2 v v^T / (v^T v), with
        // v^T v = |a_j|^2 - 2 alpha a_jj + alpha^2 = 2 alpha (alpha - a_jj)
        const double vtv = 2.0 * alpha * (alpha - A[size_t(j) * k + j]);
        A[size_t(j) * k + j] -= alpha;
        for (int q = j + 1; q < k; ++q) {
            double d = 0.0;
            for (int i = j; i < n; ++i) d += A[size_t(i) * k + j] * A[size_t(i) * k + q];
            const double f = 2.0 * d / vtv;
            for (int i = j; i < n; ++i) A[size_t(i) * k + q] -= f * A[size_t(i) * k + j];
        }
        double d = 0.0;
        for (int i = j; i < n; ++i) d += A[size_t(i) * k + j] * r[i];
        const double f = 2.0 * d / vtv;
        for (int i = j; i < n; ++i) r[i] -= f * A[size_t(i) * k + j];
        diag[j] = alpha;
    }
    for (int j = k - 1; j >= 0; --j) {
        double s = r[j];
        for (int q = j + 1; q < k; ++q) s -= A[size_t(j) * k + q] * z[q];
        z[j] = s / diag[j];
    }
    return true;
}

// One pack: returns false when the iteration limit is reached.
bool nnls(const double *B, int n, int m, const double *b, double tol, double *x) {
    bool passive[kMaxBench] = {};
    bool dependent[kMaxBench] = {};   // columns found numerically in the span of the passive ones
    double w[kMaxBench], s[kMaxBench], z[kMaxBench], res[kMaxMetrics];
    int S[kMaxBench];
    for (int i = 0; i < m; ++i) x[i] = 0.0;
    for (int outer = 0; outer < 3 * m + 10; ++outer) {
        // gradient of -1/2 ||Bx - b||^2 from the residual: w = B^T (b - B x)
        for (int r = 0; r < n; ++r) {
            double v = b[r];
            for (int q = 0; q < m; ++q) v -= B[size_t(r) * m + q] * x[q];
            res[r] = v;
        }
        int j = -1;
        for (int i = 0; i < m; ++i) {
            double g = 0.0;
            for (int r = 0; r < n; ++r) g += B[size_t(r) * m + i] * res[r];
            w[i] = g;
            if (!passive[i] && !dependent[i] && g > tol && (j < 0 || g > w[j])) j = i;
        }
        if (j < 0) return true;
        passive[j] = true;
        bool added = false;
        for (int inner = 0; inner <= m; ++inner) {
            int k = 0;
            for (int i = 0; i < m; ++i)
                if (passive[i]) S[k++] = i;
            if (!solve_passive(B, n, m, b, S, k, z)) {
                if (!passive[j]) return false;   // a subset of a solvable set failed
                // j is (numerically) in the span of the others: drop it and solve again, so
                // that x ends as the least-squares point of its passive set
                passive[j] = false;
                dependent[j] = true;
                x[j] = 0.0;
                continue;
            }
            for (int i = 0; i < m; ++i) s[i] = 0.0;
            bool positive = true;
            for (int i = 0; i < k; ++i) {
                s[S[i]] = z[i];
                if (z[i] <= 0.0) positive = false;
            }
            if (positive) {
                for (int i = 0; i < m; ++i) x[i] = s[i];
                added = passive[j];
                break;
            }
            // step from x toward s until the first passive weight reaches zero
            double alpha = 2.0;
            int qmin = -1;
            for (int i = 0; i < k; ++i) {
                const int q = S[i];
                if (s[q] <= 0.0) {
                    const double a = x[q] / (x[q] - s[q]);
                    if (a < alpha) {
                        alpha = a;
                        qmin = q;
                    }
                }
            }
            if (qmin < 0) return false;
            for (int i = 0; i < m; ++i) {
                x[i] += alpha * (s[i] - x[i]);
                // the weight that limits the step leaves exactly, whatever the rounding left
                if (passive[i] && (i == qmin || x[i] <= 0.0)) {
                    passive[i] = false;
                    x[i] = 0.0;
                }
            }
            if (inner == m) return false;
        }
        if (added)
            for (int i = 0; i < m; ++i) dependent[i] = false;
    }
    return false;
}

}  // namespace

extern "C" {

emo_status emo_pack_model(int32_t num_metrics, int32_t num_benchmarks, const float *metric_matrix,
                          int32_t num_levels, const float *bench_time, const float *bench_energy,
                          int32_t num_packs, const float *pack_metrics, float *weights,
                          float *pack_time, float *pack_energy, int32_t num_threads) {
    const int n = num_metrics, m = num_benchmarks, F = num_levels, P = num_packs;
    if (n < 1 || m < 1 || m > kMaxBench) return fail(EMO_ERR_INVALID_ARGUMENT, "need 1 <= metrics and 1 <= benchmarks <= %d", kMaxBench);
    if (F < 1 || F > 256) return fail(EMO_ERR_INVALID_ARGUMENT, "num_levels %d outside [1, 256]", F);
    if (P < 0) return fail(EMO_ERR_INVALID_ARGUMENT, "negative num_packs");
    if (!metric_matrix || !bench_time || !bench_energy) return fail(EMO_ERR_INVALID_ARGUMENT, "suite arrays are NULL");
    if (P > 0 && (!pack_metrics || !pack_time || !pack_energy)) return fail(EMO_ERR_INVALID_ARGUMENT, "pack arrays are NULL");
    for (int64_t i = 0; i < int64_t(n) * m; ++i)
        if (!std::isfinite(metric_matrix[i])) return fail(EMO_ERR_INVALID_ARGUMENT, "metric_matrix entry %lld not finite", (long long)i);
    for (int64_t i = 0; i < int64_t(m) * F; ++i)
        if (!std::isfinite(bench_time[i]) || bench_time[i] < 0.f || !std::isfinite(bench_energy[i]) || bench_energy[i] < 0.f)
            return fail(EMO_ERR_INVALID_ARGUMENT, "suite table entry %lld must be finite and >= 0", (long long)i);
    for (int64_t i = 0; i < int64_t(P) * n; ++i)
        if (!std::isfinite(pack_metrics[i])) return fail(EMO_ERR_INVALID_ARGUMENT, "pack_metrics entry %lld not finite", (long long)i);

    if (n > kMaxMetrics) return fail(EMO_ERR_INVALID_ARGUMENT, "more than %d metrics", kMaxMetrics);
    std::vector<double> Bd(size_t(n) * m);
    double colmax = 0.0;
    for (size_t i = 0; i < Bd.size(); ++i) {
        Bd[i] = double(metric_matrix[i]);
        colmax = std::max(colmax, std::fabs(Bd[i]));
    }
    std::atomic<int32_t> failed{-1};
    auto work = [&](int32_t begin, int32_t end) {
        double bd[kMaxMetrics], x[kMaxBench];
        for (int32_t p = begin; p < end; ++p) {
            double bmax = 0.0;
            for (int r = 0; r < n; ++r) {
                bd[r] = double(pack_metrics[size_t(p) * n + r]);
                bmax = std::max(bmax, std::fabs(bd[r]));
            }
            const double tol = 1e-12 * std::max(1.0, colmax) * std::max(1.0, bmax) * (n + m);
            if (!nnls(Bd.data(), n, m, bd, tol, x)) {
                int32_t expect = -1;
                failed.compare_exchange_strong(expect, p);
            }
            if (weights)
                for (int i = 0; i < m; ++i) weights[size_t(p) * m + i] = float(x[i]);
            for (int f = 0; f < F; ++f) {
                double st = 0.0, se = 0.0;
                for (int i = 0; i < m; ++i) {
                    st += x[i] * double(bench_time[size_t(i) * F + f]);
                    se += x[i] * double(bench_energy[size_t(i) * F + f]);
                }
                pack_time[size_t(p) * F + f] = float(st);
                pack_energy[size_t(p) * F + f] = float(se);
            }
        }
    };
    int T = num_threads > 0 ? num_threads : int(std::max(1u, std::thread::hardware_concurrency()));
    T = std::max(1, std::min(T, std::max(1, P / 64)));
    if (T == 1) {
        work(0, P);
    } else {
        std::vector<std::thread> pool;
        for (int t = 0; t < T; ++t)
            pool.emplace_back(work, int32_t(int64_t(P) * t / T), int32_t(int64_t(P) * (t + 1) / T));
        for (auto &th : pool) th.join();
    }
    if (failed.load() >= 0) return fail(EMO_ERR_UNSUPPORTED, "NNLS did not converge for pack %d", failed.load());
    return emo::report(EMO_OK, "");
}

}  // extern "C"
