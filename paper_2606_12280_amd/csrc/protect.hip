// Host-only selection of the protected layers (paper Section 3, "Activation-
// fragility profiling and protection"): every linear's input is profiled per
// denoising step, the layers are ranked by a fragility score, the N most
// fragile stay in bf16, and the ranking's stability over the trajectory is
// checked by the rank correlation of early and late scores.
//
// These run on the host over a few hundred numbers (the per-layer, per-step
// kurtosis that w8a8_act_moments leaves on the device, copied back by the
// caller): no kernel, no HIP call, no GPU needed. Declared in
// include/w8a8.h.
#include "../../include/w8a8.h"

#include <algorithm>
#include <cmath>
#include <numeric>
#include <stdint.h>
#include <vector>

namespace {

constexpr int64_t kMaxLayers = 1 << 20;
constexpr int64_t kMaxSteps = 1 << 20;

bool all_finite(const double *v, int64_t n) {
    for (int64_t i = 0; i < n; ++i)
        if (!std::isfinite(v[i])) return false;
    return true;
}

// 1-based ranks; entries that compare equal share the mean of the positions
// they occupy in ascending order.
std::vector<double> average_ranks(const double *v, int64_t n) {
    std::vector<int64_t> order(static_cast<size_t>(n));
    std::iota(order.begin(), order.end(), int64_t{0});
    std::stable_sort(order.begin(), order.end(),
                     [v](int64_t a, int64_t b) { return v[a] < v[b]; });
    std::vector<double> r(static_cast<size_t>(n));
    int64_t i = 0;
    while (i < n) {
        int64_t j = i;
        while (j + 1 < n && v[order[j + 1]] == v[order[i]]) ++j;
        const double rank = 0.5 * static_cast<double>(i + j) + 1.0;
        for (int64_t q = i; q <= j; ++q) r[static_cast<size_t>(order[q])] = rank;
        i = j + 1;
    }
    return r;
}

}  // namespace

extern "C" {

w8a8_status w8a8_fragility_scores(const double *kurtosis, int64_t layers, int64_t steps,
                                  int64_t step_begin, int64_t step_end, double *scores) {
    if (kurtosis == nullptr || scores == nullptr) return W8A8_ERR_NULL;
    if (layers < 1 || layers > kMaxLayers || steps < 1 || steps > kMaxSteps ||
        step_begin < 0 || step_end > steps || step_begin >= step_end)
        return W8A8_ERR_SHAPE;
    if (!all_finite(kurtosis, layers * steps)) return W8A8_ERR_UNSUPPORTED;
    const double count = static_cast<double>(step_end - step_begin);
    for (int64_t l = 0; l < layers; ++l) {
        double sum = 0.0;  // in step order
        for (int64_t s = step_begin; s < step_end; ++s) sum += kurtosis[l * steps + s];
        scores[l] = sum / count;
    }
    return W8A8_OK;
}

w8a8_status w8a8_select_protected(const double *scores, int64_t layers, int64_t n,
                                  int32_t *indices) {
    if (scores == nullptr || (indices == nullptr && n > 0)) return W8A8_ERR_NULL;
    if (layers < 1 || layers > kMaxLayers || n < 0 || n > layers) return W8A8_ERR_SHAPE;
    if (!all_finite(scores, layers)) return W8A8_ERR_UNSUPPORTED;
    std::vector<int32_t> order(static_cast<size_t>(layers));
    std::iota(order.begin(), order.end(), 0);
    // highest score first; a stable sort keeps equal scores in index order
    std::stable_sort(order.begin(), order.end(),
                     [scores](int32_t a, int32_t b) { return scores[a] > scores[b]; });
    std::copy(order.begin(), order.begin() + n, indices);
    return W8A8_OK;
}

w8a8_status w8a8_rank_correlation(const double *a, const double *b, int64_t n, double *rho) {
    if (a == nullptr || b == nullptr || rho == nullptr) return W8A8_ERR_NULL;
    if (n < 2 || n > kMaxLayers) return W8A8_ERR_SHAPE;
    if (!all_finite(a, n) || !all_finite(b, n)) return W8A8_ERR_UNSUPPORTED;
    const std::vector<double> ra = average_ranks(a, n), rb = average_ranks(b, n);
    double ma = 0.0, mb = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        ma += ra[static_cast<size_t>(i)];
        mb += rb[static_cast<size_t>(i)];
    }
    ma /= static_cast<double>(n);
    mb /= static_cast<double>(n);
    double cov = 0.0, va = 0.0, vb = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double da = ra[static_cast<size_t>(i)] - ma, db = rb[static_cast<size_t>(i)] - mb;
        cov += da * db;
        va += da * da;
        vb += db * db;
    }
    if (va == 0.0 || vb == 0.0) return W8A8_ERR_UNSUPPORTED;  // a constant vector has no ranking
    *rho = cov / std::sqrt(va * vb);
    return W8A8_OK;
}

}  // extern "C"
