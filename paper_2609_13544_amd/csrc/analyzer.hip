// The Analyzer's statistics over score series (host code; no device work):
// an operator's (mean, std) of scores across epochs and the Spearman rank
// correlation of scores with model metrics (Section IV-C), and scores in
// units of the FP64 error's score (Section V-C).
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "peat.h"

namespace {

// Average ranks (1-based) of v: sort once, then give every group of equal
// values the mean of the positions it spans.
std::vector<double> average_ranks(const std::vector<double> &v) {
    const size_t m = v.size();
    std::vector<size_t> idx(m);
    std::iota(idx.begin(), idx.end(), size_t(0));
    std::sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return v[a] < v[b]; });
    std::vector<double> r(m);
    for (size_t i = 0; i < m;) {
        size_t j = i + 1;
        while (j < m && v[idx[j]] == v[idx[i]]) ++j;
        const double rank = 0.5 * (double)(i + 1 + j);    // mean of positions i+1 .. j
        for (size_t k = i; k < j; ++k) r[idx[k]] = rank;
        i = j;
    }
    return r;
}

}  // namespace

extern "C" {

int peat_series_stats(const double *x, int64_t n, peat_series_t *out) {
    if (!out || n < 0 || (n > 0 && !x)) return PEAT_EINVAL;
    peat_series_t r{0, NAN, NAN, NAN, NAN, NAN};
    // two passes with extended-precision (x87 80-bit) accumulators
    long double sum = 0;
    for (int64_t i = 0; i < n; ++i) {
        const double v = x[i];
        if (std::isnan(v)) continue;
        if (r.count == 0 || v < r.min) r.min = v;
        if (r.count == 0 || v > r.max) r.max = v;
        r.count += 1;
        sum += v;
    }
    if (r.count > 0) r.mean = (double)(sum / (long double)r.count);
    if (r.count > 1) {
        long double ss = 0;
        for (int64_t i = 0; i < n; ++i) {
            if (std::isnan(x[i])) continue;
            const long double d = (long double)x[i] - (long double)r.mean;
            ss += d * d;
        }
        r.var = (double)(ss / (long double)(r.count - 1));
        r.std = std::sqrt(r.var);
    }
    *out = r;
    return PEAT_OK;
}

int peat_normalize_scores(const double *scores, const double *units, int64_t n, double *out) {
    if (n < 0 || (n > 0 && (!scores || !units || !out))) return PEAT_EINVAL;
    for (int64_t i = 0; i < n; ++i) out[i] = scores[i] / units[i];
    return PEAT_OK;
}

int peat_spearman(const double *x, const double *y, int64_t n, double *rho) {
    if (!rho || n < 0 || (n > 0 && (!x || !y))) return PEAT_EINVAL;
    std::vector<double> xs, ys;
    for (int64_t i = 0; i < n; ++i) {
        if (std::isnan(x[i]) || std::isnan(y[i])) continue;
        xs.push_back(x[i]);
        ys.push_back(y[i]);
    }
    *rho = NAN;
    const size_t m = xs.size();
    if (m < 2) return PEAT_OK;
    const std::vector<double> rx = average_ranks(xs), ry = average_ranks(ys);
    const double mean = 0.5 * (double)(m + 1);
    long double sxy = 0, sxx = 0, syy = 0;
    for (size_t i = 0; i < m; ++i) {
        const long double dx = rx[i] - mean, dy = ry[i] - mean;
        sxy += dx * dy;
        sxx += dx * dx;
        syy += dy * dy;
    }
    if (sxx > 0 && syy > 0) *rho = (double)(sxy / std::sqrt(sxx * syy));
    return PEAT_OK;
}

}  // extern "C"
