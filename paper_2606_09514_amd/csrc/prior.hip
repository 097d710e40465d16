// Offline prior normalisation (App. B "Prior Indicators and Normalization",
// fused by Eq. 2): raw per-layer importance indicators to the standardised
// prior p~ that buddy_dm_weights.prior takes.  Host code, float64 inside.
#include <math.h>
#include <stdlib.h>
#include <string.h>
#include <vector>
#include <algorithm>

#include "../../include/buddy.h"

namespace {

constexpr double kEps = 1e-6;

// Quantile of sorted values with linear interpolation between order statistics.
double quantile(const std::vector<double>& sorted, double q) {
    const double at = q * (double)(sorted.size() - 1);
    const size_t lo = (size_t)floor(at);
    const size_t hi = lo + 1 < sorted.size() ? lo + 1 : lo;
    return sorted[lo] + (at - (double)lo) * (sorted[hi] - sorted[lo]);
}

}  // namespace

extern "C" buddy_status buddy_prior_normalize(const float* raw, int32_t n, int32_t kind,
                                              float winsor, float* prior_out) {
    if (!raw || !prior_out || n < 1) return BUDDY_EINVAL;
    if (kind != BUDDY_PRIOR_DELTA_PPL && kind != BUDDY_PRIOR_TAYLOR && kind != BUDDY_PRIOR_COSINE)
        return BUDDY_EINVAL;
    if (!(winsor >= 0.f) || !isfinite(winsor)) return BUDDY_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        if (!isfinite(raw[i])) return BUDDY_EINVAL;

    // (i) larger means more important; (ii) log(1 + x) for the heavy-tailed kinds
    std::vector<double> x(n);
    for (int32_t i = 0; i < n; ++i) {
        const double r = raw[i];
        x[i] = kind == BUDDY_PRIOR_COSINE ? 1.0 - r : log1p(r > 0.0 ? r : 0.0);
    }
    // (iii) robust z-score over the layers, optionally winsorised at +-winsor
    std::vector<double> s(x);
    std::sort(s.begin(), s.end());
    const double med = quantile(s, 0.5), iqr = quantile(s, 0.75) - quantile(s, 0.25);
    std::vector<double> z(n);
    for (int32_t i = 0; i < n; ++i) {
        z[i] = (x[i] - med) / (iqr + kEps);
        if (winsor > 0.f) z[i] = std::min(std::max(z[i], -(double)winsor), (double)winsor);
    }
    // (iv) rank normalisation u = (1 + rank) / (n + 1), ties at their mean rank
    std::vector<double> u(n);
    for (int32_t i = 0; i < n; ++i) {
        int32_t below = 0, equal = 0;
        for (int32_t j = 0; j < n; ++j) {
            below += z[j] < z[i];
            equal += z[j] == z[i];
        }
        u[i] = (1.0 + below + 0.5 * (equal - 1)) / (double)(n + 1);
    }
    // Eq. 2: p~ = (u - mean) / (population std + eps)
    double mean = 0.0;
    for (double v : u) mean += v;
    mean /= n;
    double var = 0.0;
    for (double v : u) var += (v - mean) * (v - mean);
    const double sd = sqrt(var / n);
    for (int32_t i = 0; i < n; ++i) prior_out[i] = (float)((u[i] - mean) / (sd + kEps));
    return BUDDY_OK;
}
